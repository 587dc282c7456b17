#!/usr/bin/env python3
"""Benchmark of the RippleKV sensitivity profile on one MI355X.

Default workload: the Llama-3-8B-shaped decoder at long context (32 layers,
d_model 4096, 32 query / 8 KV heads of 128, SwiGLU 14336, vocab 128256, rotary
theta 5e5, bf16) on 2 calibration sequences of 32768 Zipf(1.1) tokens with
alpha in {0.05, 0.1, 0.2}.  One step is the whole profiling path of Algorithm 1
for one (sequence, alpha) pair: the clean reference pass, the 32 resumed
perturbed passes (prefix reuse), the fused LM-head + KL, the window and
calibration means, then the budget mapping for every ratio and global budget;
steps cycle over the six pairs.  With ``--workload NAME`` (and ``--step-unit
profile``) one step is the whole profile of that workload instead.  Inputs
(random-init weights, tokens) are synthetic and resident in HBM before timing.

Prints one JSON line: perturbed token-layers per second (whole job), the
roofline of the dominant kernel measured live with HIP events over the timed
steps, and the CPU oracle's rate on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                    [--workload NAME] [--step-unit auto|pair|profile]
                    [--window N | --snapkv | --damage]
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
# profiles/).  Keyed by (family, workload, resumed passes per launch); valid only
# while the family's kernel sources hash to the recorded value, so a changed
# kernel or launch shape reports null until re-measured.
TRAFFIC = {
    ("gemm_gate_up", "gpt2s-bf16", 1): {"bytes_per_launch": 327091576, "fetch_bytes": 226428280,
                                     "write_bytes": 100663296, "sources": "5138ba9bfc0b0ac1"},
    ("gemm_gate_up", "llama3-8b-long-bf16", 1): {"bytes_per_launch": 12252797172, "fetch_bytes": 11313273076,
                                                 "write_bytes": 939524096, "sources": "3637cd35c57e36e6"},
    ("attention", "llama3-8b-long-bf16", 1): {"bytes_per_launch": 1677633940, "fetch_bytes": 1409141478,
                                              "write_bytes": 268492462, "sources": "e2f55bc60551caaf"},
}
FAMILY_SOURCES = {
    "gemm": ["paper_2608_08684_amd/csrc/gemm.hip", "paper_2608_08684_amd/csrc/mfma_tile.h"],
    "attention": ["paper_2608_08684_amd/csrc/attention.hip"],
    "lm_kl": ["paper_2608_08684_amd/csrc/lm_kl.hip", "paper_2608_08684_amd/csrc/mfma_tile.h"],
}
FAMILY_KERNEL = {"gemm_gate_up": "EpiSwiGLU", "gemm_qkv": "EpiRope", "lm_kl": "lm_kl_kernel",
                 "attention": "attn_bf16_kernel"}


def sources_hash(family: str) -> str:
    """Digest of the kernel sources of a family (gemm_* share the GEMM sources)."""
    import hashlib
    h = hashlib.sha256()
    for rel in FAMILY_SOURCES["gemm" if family.startswith("gemm") else family]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_of(family: str, workload: str, passes_per_launch: int = 1):
    """Recorded HBM bytes per launch of a family, or None once its sources changed."""
    rec = TRAFFIC.get((family, workload, passes_per_launch))
    return rec["bytes_per_launch"] if rec is not None and rec["sources"] == sources_hash(family) else None


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
            "fetch_scale": f_scale, "write_scale": w_scale, "sources": sources_hash(family)}


# kernel families of the profile, by a substring of the kernel name (first match wins)
FAMILIES = [("gemm_gate_up", "EpiSwiGLU"), ("gemm_qkv", "EpiRope"), ("gemm_o_down", "EpiResidual"),
            ("lm_kl", "lm_kl_kernel"), ("lm_lse", "lm_lse_kernel"), ("attention", "attn_bf16_kernel"),
            ("rmsnorm", "rmsnorm_kernel"), ("noise", "value_noise_kernel"), ("kl_merge", "kl_merge_kernel"),
            ("kl_logits", "kl_logits_kernel"), ("lm_logits", "EpiStoreF32"),
            ("local_response", "local_response_kernel")]


def family_of(name: str):
    for fam, key in FAMILIES:
        if key in name:
            return fam
    return None


def derive_counters(dirs):
    """Per kernel family, from rocprofv3 --pmc csv directories of this benchmark:
    mean counters per dispatch and mean dispatch duration, with MFMA-busy share
    of the CU-busy cycles (SQ_VALU_MFMA_BUSY_CYCLES counts per SIMD, four per CU),
    the share of wave cycles spent waiting, and the clock implied by
    GRBM_GUI_ACTIVE (summed over the 8 XCDs) over the duration, which is only
    meaningful for dispatches much longer than the profiler's own overhead (ms,
    not us).  Prints a markdown table."""
    import csv
    import glob
    from collections import defaultdict
    vals = defaultdict(lambda: defaultdict(list))
    durs = defaultdict(list)
    ids = defaultdict(lambda: defaultdict(set))   # dispatches per family and counter run
    for d in dirs:
        for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
            for r in csv.DictReader(open(f)):
                fam = family_of(r["Kernel_Name"])
                if fam is None:
                    continue
                vals[fam][r["Counter_Name"]].append(float(r["Counter_Value"]))
                durs[fam].append((float(r["End_Timestamp"]) - float(r["Start_Timestamp"])))
                ids[fam][d].add(r["Dispatch_Id"])
    mean = lambda x: sum(x) / len(x) if x else float("nan")
    print("| family | dispatches | avg us | MFMA busy / CU busy | waiting / wave cycles | clock GHz |")
    print("|---|---|---|---|---|---|")
    for fam, _ in FAMILIES:
        if fam not in vals:
            continue
        v = {k: mean(x) for k, x in vals[fam].items()}
        n = max(len(x) for x in ids[fam].values())
        dur = mean(durs[fam])
        mf = v.get("SQ_VALU_MFMA_BUSY_CYCLES", float("nan")) / (4.0 * v.get("SQ_BUSY_CU_CYCLES", float("nan")))
        wt = v.get("SQ_WAIT_ANY", float("nan")) / v.get("SQ_WAVE_CYCLES", float("nan"))
        ck = v.get("GRBM_GUI_ACTIVE", float("nan")) / 8.0 / dur
        print(f"| {fam} | {n} | {dur / 1e3:.1f} | {mf:.3f} | {wt:.3f} | {ck:.2f} |")
    # LDS pass (when collected): the share of cycles the LDS of a CU is busy with
    # indexed accesses (SQ_LDS_IDX_ACTIVE over GRBM_GUI_ACTIVE per XCD x 256 CUs),
    # bank-conflict cycles per busy cycle, and the share of wave cycles spent
    # waiting to issue LDS instructions
    if not any("SQ_LDS_IDX_ACTIVE" in vals[f] for f in vals):
        return
    print()
    print("| family | LDS busy / elapsed | bank conflicts / LDS busy | waiting on LDS issue / wave cycles |")
    print("|---|---|---|---|")
    for fam, _ in FAMILIES:
        if fam not in vals or "SQ_LDS_IDX_ACTIVE" not in vals[fam]:
            continue
        v = {k: mean(x) for k, x in vals[fam].items()}
        busy = v["SQ_LDS_IDX_ACTIVE"] / (v.get("GRBM_GUI_ACTIVE", float("nan")) / 8.0 * 256.0)
        conf = v.get("SQ_LDS_BANK_CONFLICT", float("nan")) / v["SQ_LDS_IDX_ACTIVE"] if v["SQ_LDS_IDX_ACTIVE"] else 0.0
        wl = v.get("SQ_WAIT_INST_LDS", float("nan")) / v.get("SQ_WAVE_CYCLES", float("nan"))
        print(f"| {fam} | {busy:.3f} | {conf:.4f} | {wl:.3f} |")


def derive_traffic_table(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir):
    """Per kernel family: HBM bytes per dispatch (FETCH_SIZE and WRITE_SIZE scaled
    by the 1 GiB copy calibration) and the rate over the mean dispatch duration
    of the same counter runs.  Prints a markdown table."""
    import csv
    import glob
    from collections import defaultdict

    def per_family(d, calib):
        out, durs = defaultdict(list), defaultdict(list)
        for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
            for r in csv.DictReader(open(f)):
                fam = "copy" if calib and "copyBuffer" in r["Kernel_Name"] else family_of(r["Kernel_Name"])
                if fam is None:
                    continue
                out[fam].append(float(r["Counter_Value"]) * 1024.0)
                durs[fam].append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
        return ({k: sum(x) / len(x) for k, x in out.items()}, {k: sum(x) / len(x) for k, x in durs.items()})

    cf, _ = per_family(copy_fetch_dir, True)
    cw, _ = per_family(copy_write_dir, True)
    fs, ws = float(1 << 30) / cf["copy"], float(1 << 30) / cw["copy"]
    fetch, df = per_family(fetch_dir, False)
    write, dw = per_family(write_dir, False)
    print(f"| family | HBM read MB | HBM write MB | avg us | GB/s | of 8 TB/s |  (FETCH x {fs:.3f}, WRITE x {ws:.3f})")
    print("|---|---|---|---|---|---|")
    for fam, _ in FAMILIES:
        if fam not in fetch or fam not in write:
            continue
        rd, wr = fetch[fam] * fs, write[fam] * ws
        dur = (df[fam] + dw[fam]) / 2.0
        gbs = (rd + wr) / dur
        print(f"| {fam} | {rd / 1e6:.1f} | {wr / 1e6:.1f} | {dur / 1e3:.1f} | {gbs:.0f} | {gbs / HBM_PEAK_GBS:.2f} |")


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


def step_flops(cfg, lens, layers, alphas, P: int = 0, local: bool = False) -> float:
    """Algorithmic MFMA work of one profile call: the clean pass (every layer over
    every row, plus the clean LM head over the evaluated rows) and, per pass (alpha, l), layers l .. L-1
    over the evaluated rows with their causal attention plus the perturbed LM
    head (the clean logits the fused kernel recomputes are not counted).  In the
    cached-window mode the evaluated rows are [P, T_i) attending to the whole
    prefix; with the layer-local signal a pass runs layer l only, and no LM head."""
    d, H, Hkv, dh, ff, V, L = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff, cfg.vocab, cfg.n_layers
    lin = 2.0 * d * (H + 2 * Hkv) * dh + 2.0 * H * dh * d + 2.0 * d * 2 * ff + 2.0 * ff * d   # per row and layer

    def attn(q0):   # causal attention of query rows [q0, T) of every sequence, one layer
        return sum(4.0 * H * dh * ((T * (T + 1) - q0 * (q0 + 1)) / 2) for T in lens)
    rows_all, rows_eval = sum(lens), sum(T - P for T in lens)
    clean = L * (lin * rows_all + attn(0)) + (0.0 if local else 2.0 * rows_eval * d * V)
    per_layer_pass = lin * rows_eval + attn(P)
    if local:
        passes = len(alphas) * len(layers) * per_layer_pass
    else:
        passes = len(alphas) * sum((L - l) * per_layer_pass + 2.0 * rows_eval * d * V for l in layers)
    return clean + passes


def cpu_baseline_window(w, W, toks, window: int):
    """Oracle cached-window profile of sequence 0 (prefix prefill and window
    reference included), every layer, the largest alpha."""
    from oracle import model as OM
    from oracle import profile as OPR
    from fixtures import f32_weights
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


def cpu_sample(cfg):
    """The oracle's bounded sample of a workload: (tokens of sequence 0, layers).
    Every layer of a 2048-token prefix for the small models; for the 7-8B shapes
    (about 0.44 GFLOP per token and layer) a 256-token prefix and the last and
    middle layers, so the host run stays within tens of seconds."""
    if cfg.d_model <= 1024:
        return 2048, list(range(cfg.n_layers))
    return 256, [cfg.n_layers - 1, cfg.n_layers // 2]


def cpu_baseline(w, W, toks, local: bool = False):
    """Oracle (as it stands) on a bounded sample: the first tokens of sequence 0
    (a causal prefix computes exactly the same per-position values) and a set of
    layers (cpu_sample), the largest alpha, clean pass included (the layer-local
    signal with `local`)."""
    from oracle import model as OM
    from oracle import profile as OPR
    from fixtures import f32_weights  # exact fp32 view of the bf16 weights
    cfg = w.model
    prefix, layers = cpu_sample(cfg)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0][:prefix]
    alpha = max(w.alphas)
    t0 = time.perf_counter()
    st = OM.clean_pass(m, t)
    one = OPR.local_profile_layer if local else OPR.profile_layer
    for l in layers:
        one(m, st, t, 0, l, OPR.PerturbParams(alpha))
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    n = len(t) * len(layers)
    which = f"all {cfg.n_layers} layers" if len(layers) == cfg.n_layers else f"layers {layers}"
    return {"value": n / dt, "unit": "perturbed token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {len(t)} tokens of sequence 0, {which}, alpha={alpha}, float32 oracle"
                      f"{' (layer-local signal)' if local else ''}: {dt:.1f} s for {n} token-layers (clean pass "
                      f"included)"}


SNAP_WINDOW, SNAP_KERNEL, SNAP_RHO, SNAP_RATIO = 32, 7, 0.2, 2.0


def snapkv_budgets(w, L: int):
    """Per-sequence, per-layer budgets: B_i = rho T_i L (Eq. global-budget with a
    retention ratio rho) split by the allocation half of Algorithm 1 over a fixed
    decreasing profile s_l = 1 / (1 + l)."""
    import paper_2608_08684_amd as rk
    s = [1.0 / (1.0 + l) for l in range(L)]
    return np.array([rk.layer_budgets(s, int(round(SNAP_RHO * T * L)), SNAP_RATIO)[1] for T in w.lengths()],
                    dtype=np.int64)


def snapkv_bytes(cfg, lens, budgets, obs: int):
    """Algorithmic HBM bytes per layer of the two kernel families (averaged over
    layers): scores read every Key twice (statistics, then votes), the observation
    queries once and write the votes; select reads the votes, reads and writes the
    retained Keys and Values and writes their positions."""
    R, n = int(sum(lens)), len(lens)
    L, Hkv, H, dh = cfg.n_layers, cfg.n_kv_heads, cfg.n_heads, cfg.head_dim
    pre = R - n * obs
    scores = 2 * R * Hkv * dh * 2 + n * obs * H * dh * 2 + Hkv * pre * 4
    kept = sum(min(max(int(b), 0), T) for T, row in zip(lens, budgets) for b in row) / L
    select = Hkv * pre * 4 + kept * Hkv * (4 * dh * 2 + 4)
    return scores, select


def cpu_baseline_snapkv(cfg, layers: int = 6):
    """Oracle SnapKV selection of one 8192-token sequence of the same shape, the
    first `layers` layers of a fixtures cache state."""
    import fixtures as F
    from oracle import snapkv as OS
    T, obs = 8192, SNAP_WINDOW
    H, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    kv, q = F.make_kv_state(layers, [T], H, Hkv, dh, obs, seed_id=99)
    p = OS.SnapParams(obs_window=obs, pool_kernel=SNAP_KERNEL)
    b = int(round(SNAP_RHO * T))
    t0 = time.perf_counter()
    for l in range(layers):
        k = F.bf16_to_f32(kv[l, :, : Hkv * dh]).astype(np.float64).reshape(T, Hkv, dh)
        v = F.bf16_to_f32(kv[l, :, Hkv * dh:]).astype(np.float64).reshape(T, Hkv, dh)
        qq = np.zeros((T, H, dh))
        qq[T - obs:] = F.bf16_to_f32(q[l]).astype(np.float64).reshape(obs, H, dh) * (np.sqrt(dh) / 1.4426950408889634)
        OS.compress_layer(qq, k, v, b, p)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    return {"value": T * layers / dt, "unit": "prompt token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"one {T}-token sequence of the same shape, {layers} layers, b = {b}, float64 oracle: "
                      f"{dt:.1f} s"}


def snapkv_main(args):
    """SnapKV selection with the per-layer budgets (the budgets' consumer) on the
    Llama-3-8B shape: 4 x 8192-token prompts, 32 layers, 32 query / 8 KV heads of
    128, observation window 32, max pooling 7, budgets from a 20% retention."""
    import torch
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens as make_batch
    w = F.get_workload("llama3-8b-bf16")
    cfg = w.model
    L, H, Hkv, dh = cfg.n_layers, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    lens = w.lengths()
    obs = SNAP_WINDOW
    t0 = time.perf_counter()
    # the selection reads only the model's shape; one placeholder buffer stands in for the weights
    ph = torch.zeros(256, dtype=torch.uint8, device="cuda")
    model = rk.Model(cfg, {"tok_emb": ph, "lm_head": ph, "final_norm": ph,
                           **{k: [ph] * L for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "mlp_norm")}})
    batch = make_batch([np.zeros(T, dtype=np.int32) for T in lens])
    R = batch.rows
    # prompt caches: two fixtures layers, repeated over the 32 layers
    kv2, q2 = F.make_kv_state(2, lens, H, Hkv, dh, obs, seed_id=7)
    state = torch.empty(model.snapkv_state_size(R, len(lens), obs), dtype=torch.uint8, device="cuda")
    kvl = R * 2 * Hkv * dh * 2
    ql = len(lens) * obs * H * dh * 2
    q_off = (L * kvl + 255) // 256 * 256
    for l in range(L):
        state[l * kvl:(l + 1) * kvl] = torch.from_numpy(kv2[l % 2].reshape(-1).view(np.uint8)).cuda()
        state[q_off + l * ql:q_off + (l + 1) * ql] = torch.from_numpy(q2[l % 2].reshape(-1).view(np.uint8)).cuda()
    del kv2, q2
    budgets = snapkv_budgets(w, L)
    total, _ = rk.snapkv_layout(batch, L, budgets)
    pos = torch.empty(Hkv * total, dtype=torch.int32, device="cuda")
    ko = torch.empty(Hkv * total, dh, dtype=torch.int16, device="cuda")
    vo = torch.empty_like(ko)
    ws = torch.empty(model.snapkv_workspace_size(R, len(lens), obs), dtype=torch.uint8, device="cuda")
    log(f"SnapKV inputs ready in {time.perf_counter() - t0:.1f} s")

    def step():
        model.snapkv_compress(batch, budgets, state, pos, ko, vo, ws, obs_window=obs, pool_kernel=SNAP_KERNEL,
                              pooling=rk.RK_POOL_MAX)

    fams = ("snap_scores", "snap_select")
    for k in range(args.warmup):
        step()
    torch.cuda.synchronize()
    fam_ms = {f: 0.0 for f in fams}
    fam_n = {f: 0 for f in fams}
    fam_steps = {f: 0 for f in fams}
    t0 = time.perf_counter()
    for k in range(args.steps):
        f = fams[k % 2]                 # alternate the timed family step by step
        rk.timing_begin(f)
        step()
        n, ms = rk.timing_end()
        fam_n[f] += n
        fam_ms[f] += ms
        fam_steps[f] += 1
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    value = R * L / (ms_per_step / 1e3)
    # algorithmic bytes per launch = bytes of every layer / launches per call
    per_layer = dict(zip(fams, snapkv_bytes(cfg, lens, budgets, obs)))
    per_launch = {f: per_layer[f] * L / (fam_n[f] / max(fam_steps[f], 1)) if fam_n[f] else 0.0 for f in fams}
    avg = {f: fam_ms[f] / max(fam_n[f], 1) for f in fams}
    step_ms = {f: fam_ms[f] / max(fam_steps[f], 1) for f in fams}
    dom = max(fams, key=lambda f: step_ms[f])
    achieved = per_launch[dom] / (avg[dom] / 1e3) / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": dom, "launches": fam_n[dom],
            "avg_ms": round(avg[dom], 4), "bytes_per_launch": int(per_launch[dom]),
            "other": {f: {"avg_ms": round(avg[f], 4), "bytes_per_launch": int(per_launch[f]),
                          "GB/s": round(per_launch[f] / (avg[f] / 1e3) / 1e9, 1)} for f in fams if f != dom}}
    log(f"{dom}: {fam_n[dom]} launches, avg {avg[dom]:.4f} ms, {achieved:.0f} GB/s")
    res = {
        "metric": "prompt token-layers/s (SnapKV selection with per-layer budgets)",
        "value": round(value, 1), "unit": "token-layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (fixtures cache state: N(0,1) keys and values "
                                                       "with heavy hitters, observation queries)",
        "config": {"workload": f"llama3-8b-bf16 SnapKV: {L}L {H}q/{Hkv}kv x {dh}; {len(lens)}x{max(lens)} tokens; "
                               f"window {obs}, max pooling {SNAP_KERNEL}; budgets rho {SNAP_RHO}, r {SNAP_RATIO} "
                               f"over s_l = 1/(1+l); {total} kept positions per KV head"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_snapkv(cfg)
    print(json.dumps(res), flush=True)


DMG_RHO, DMG_OBS = 0.2, 32


def cpu_baseline_damage(w, W, toks, P: int, b: int):
    """Oracle isolated compression damage of sequence 0 (window reference
    included), every layer, b retained prompt positions per KV head drawn by
    fixtures (the oracle's cost does not depend on which positions are kept)."""
    import fixtures as F
    from oracle import damage as OD
    from oracle import model as OM
    from oracle import profile as OPR
    from fixtures import f32_weights
    cfg = w.model
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0]
    pos = F.random_keep(1, cfg.n_kv_heads, P, b, seed_id=5)[0]
    t0 = time.perf_counter()
    ws = OPR.window_clean_state(m, t, P)
    for l in range(cfg.n_layers):
        OD.damage_layer(m, ws, l, list(pos))
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    n = (len(t) - P) * cfg.n_layers
    return {"value": n / dt, "unit": "window token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"sequence 0 (prompt {P}, window {len(t) - P}), all {cfg.n_layers} layers, {b} kept positions "
                      f"per KV head, float32 oracle: {dt:.1f} s (window reference included)"}


def cpu_baseline_policy(w, W, toks, P: int, budgets):
    """Oracle whole-policy damage of sequence 0 (window reference included): every
    layer compressed to its budget, positions drawn by fixtures (the oracle's cost
    does not depend on which positions are kept)."""
    import fixtures as F
    from oracle import damage as OD
    from oracle import model as OM
    from oracle import profile as OPR
    from fixtures import f32_weights
    cfg = w.model
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0]
    keep = [list(F.random_keep(1, cfg.n_kv_heads, P, int(b), seed_id=20 + l)[0]) for l, b in enumerate(budgets)]
    t0 = time.perf_counter()
    ws = OPR.window_clean_state(m, t, P)
    OD.policy_damage(m, ws, keep)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    n = (len(t) - P) * cfg.n_layers
    return {"value": n / dt, "unit": "window token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"sequence 0 (prompt {P}, window {len(t) - P}), all {cfg.n_layers} layers compressed to the "
                      f"RippleKV budgets, float32 oracle: {dt:.1f} s (window reference included)"}


def policy_main(args):
    """The damage of whole per-layer budget policies on the GPT-2-small-shaped
    workload: the cached-window sensitivity profile of the batch gives RippleKV
    budgets (ratio 2, the same total as SnapKV's uniform b = 20% of the prompt at
    every layer); SnapKV selects each policy's positions on the prompts; one step
    = the sweep over the ratio (1 = uniform, 1.5, 2, 4, 8) in one
    rk_policy_damage_group call (the window evaluated with every layer's prompt
    cache compressed, each policy's pass batched with the others, fused LM head
    + KL against the full-cache window) and the batch means.  The time of a
    single-policy rk_policy_damage call is reported beside it."""
    import torch
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens as make_batch, upload_weights
    w = F.get_workload(args.workload)
    cfg = w.model
    L, Hkv, dh = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    window = args.window if args.window > 0 else 256
    lens = w.lengths()
    P = min(lens) - window
    b = int(round(DMG_RHO * P))
    t0 = time.perf_counter()
    W = F.make_weights(cfg)
    model = rk.Model(cfg, upload_weights(W))
    toks = F.make_tokens(w)
    batch = make_batch(toks)
    rows = batch.rows
    Rw = sum(T - P for T in lens)
    state = torch.empty(model.window_state_size(rows), dtype=torch.uint8, device="cuda")
    ws = torch.empty(model.workspace_size(rows, L, rk.RK_FLAG_CACHED_WINDOW), dtype=torch.uint8, device="cuda")
    model.window_reference(batch, P, state, ws)
    s_out = torch.empty(1, L, dtype=torch.float32, device="cuda")
    pws = torch.empty(model.workspace_size(rows, L, rk.RK_WS_CLEAN_STATE | rk.RK_FLAG_CACHED_WINDOW),
                      dtype=torch.uint8, device="cuda")
    model.sensitivity_profile(batch, list(range(L)), [max(w.alphas)], s_out, pws, rows, L, window_start=P,
                              flags=rk.RK_FLAG_CACHED_WINDOW)
    s_prof = s_out.cpu().numpy()[0].astype(np.float64)
    del pws
    def ripple_budgets(r):
        _, bl = rk.layer_budgets(s_prof, b * L, r)
        return [max(1, min(int(x), P)) for x in bl]
    ripple = ripple_budgets(2.0)
    sweep_r = (1.5, 4.0, 8.0)
    pb = make_batch([t[:P] for t in toks])
    sst = torch.empty(model.snapkv_state_size(pb.rows, pb.n_seqs, DMG_OBS), dtype=torch.uint8, device="cuda")
    sws = torch.empty(model.snapkv_workspace_size(pb.rows, pb.n_seqs, DMG_OBS), dtype=torch.uint8, device="cuda")
    model.snapkv_prefill(pb, DMG_OBS, sst, sws)
    policies = {}
    for name, bl in [("uniform", [b] * L), ("ripplekv", ripple)] + [(f"r{r}", ripple_budgets(r)) for r in sweep_r]:
        # ratio 1 gives the uniform budgets (up to rounding): the uniform policy stands for it
        budgets = np.tile(np.asarray(bl, dtype=np.int64), (pb.n_seqs, 1))
        total, offs = rk.snapkv_layout(pb, L, budgets)
        pos = torch.empty(Hkv * total, dtype=torch.int32, device="cuda")
        ko = torch.empty(Hkv * total, dh, dtype=torch.int16, device="cuda")
        vo = torch.empty_like(ko)
        model.snapkv_compress(pb, budgets, sst, pos, ko, vo, sws, obs_window=DMG_OBS)
        policies[name] = (pos, [int(offs[l]) * Hkv for l in range(L)], int(offs[L]) * Hkv, bl)
        del ko, vo
    del sst, sws
    ratios = (1.0, 1.5, 2.0, 4.0, 8.0)
    names = ["uniform", "r1.5", "ripplekv", "r4.0", "r8.0"]
    group = [policies[n] for n in names]
    G = len(group)
    d_out = torch.empty(G, batch.n_seqs, dtype=torch.float32, device="cuda")
    log(f"policy inputs ready in {time.perf_counter() - t0:.1f} s (prompt {P}, window {window}, uniform b = {b}, "
        f"RippleKV budgets {ripple})")

    def run():
        model.policy_damage_group(batch, P, group, state, d_out, ws)
        return d_out.mean(dim=1).cpu().numpy().astype(np.float64)     # synchronises

    # the single-policy call for the RippleKV policy, once (its time is reported beside the group's)
    pos, loff, stride, bl = policies["ripplekv"]
    d1 = torch.empty(batch.n_seqs, dtype=torch.float32, device="cuda")
    model.policy_damage(batch, P, pos, loff, stride, bl, state, d1, ws)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(5):
        model.policy_damage(batch, P, pos, loff, stride, bl, state, d1, ws)
    torch.cuda.synchronize()
    single_ms = (time.perf_counter() - t1) * 1e3 / 5
    for _ in range(args.warmup):
        rk.timing_begin(args.family)
        run()
        rk.timing_end()
    torch.cuda.synchronize()
    launches, fam_ms = 0, 0.0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        rk.timing_begin(args.family)
        D = run()
        n, ms = rk.timing_end()
        launches += n
        fam_ms += ms
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    value = Rw * L * G / (ms_per_step / 1e3)
    avg = fam_ms / max(launches, 1)
    if args.family == "lm_kl":
        flops = family_flops(args.family, cfg, Rw * G, 1) * args.steps / max(launches, 1)
    else:   # every policy's pass runs every layer once over the window rows
        flops = family_flops(args.family, cfg, Rw * L * G, 1) * args.steps / max(launches, 1)
    achieved = flops / (avg / 1e3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": None, "kernel": args.family,
            "launches": launches, "avg_ms": round(avg, 4), "flop_per_launch": flops}
    sweep = {str(r): float(x) for r, x in zip(ratios, D)}
    log(f"{args.family}: {launches} launches, avg {avg:.4f} ms, {achieved:.1f} TFLOP/s; damage by ratio {sweep}; "
        f"one policy alone {single_ms:.3f} ms")
    res = {
        "metric": "window token-layers/s (whole-policy compressed-cache window evaluation)",
        "value": round(value, 1), "unit": "token-layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (random-init N(0,0.02) weights, Zipf(1.1) tokens)",
        "config": {"workload": f"{w.name} budget policies: {L}L d{cfg.d_model} {cfg.n_heads}x{dh}; "
                               f"{batch.n_seqs}x{max(lens)} tokens, prompt {P} + window {window}; SnapKV selection "
                               f"(window {DMG_OBS}, max pooling 7) with RippleKV budgets at ratios {list(ratios)} "
                               f"(ratio 1 = uniform b = {b}; same total), every layer compressed at once; one step = "
                               f"the {G} policies in one rk_policy_damage_group call",
                   "ripplekv_budgets": ripple, "damage_by_ratio": sweep,
                   "single_policy_ms": round(single_ms, 3)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_policy(w, W, toks, P, ripple)
    print(json.dumps(res), flush=True)


def damage_main(args):
    """Isolated single-layer compression damage (Section 2) of every layer on the
    GPT-2-small-shaped workload: the prompt [0, P) of each sequence compressed by
    SnapKV with the same budget b at every layer, one layer at a time, the window
    [P, T) evaluated against the caches; then Spearman's rho of the damage profile
    against the cached-window sensitivity profile.  One step = the damage of every
    layer for all sequences (one rk_compression_damage_layers call: each layer's
    pass joins the batch at that layer) plus the rank correlation."""
    import torch
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens as make_batch, upload_weights
    w = F.get_workload(args.workload)
    cfg = w.model
    L, Hkv, dh = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    window = args.window if args.window > 0 else 256
    lens = w.lengths()
    P = min(lens) - window
    b = int(round(DMG_RHO * P))
    t0 = time.perf_counter()
    W = F.make_weights(cfg)
    model = rk.Model(cfg, upload_weights(W))
    toks = F.make_tokens(w)
    batch = make_batch(toks)
    rows = batch.rows
    # the prompts' caches and the window reference
    state = torch.empty(model.window_state_size(rows), dtype=torch.uint8, device="cuda")
    ws = torch.empty(model.workspace_size(rows, L, rk.RK_FLAG_CACHED_WINDOW), dtype=torch.uint8, device="cuda")
    model.window_reference(batch, P, state, ws)
    # SnapKV on the prompts with the same budget at every layer (the base compressor)
    pb = make_batch([t[:P] for t in toks])
    sst = torch.empty(model.snapkv_state_size(pb.rows, pb.n_seqs, DMG_OBS), dtype=torch.uint8, device="cuda")
    sws = torch.empty(model.snapkv_workspace_size(pb.rows, pb.n_seqs, DMG_OBS), dtype=torch.uint8, device="cuda")
    model.snapkv_prefill(pb, DMG_OBS, sst, sws)
    budgets = np.full((pb.n_seqs, L), b, dtype=np.int64)
    total, _ = rk.snapkv_layout(pb, L, budgets)
    pos = torch.empty(Hkv * total, dtype=torch.int32, device="cuda")
    ko = torch.empty(Hkv * total, dh, dtype=torch.int16, device="cuda")
    vo = torch.empty_like(ko)
    model.snapkv_compress(pb, budgets, sst, pos, ko, vo, sws, obs_window=DMG_OBS)
    del sst, sws, ko, vo
    # the cached-window sensitivity profile the damage is ranked against
    s_out = torch.empty(1, L, dtype=torch.float32, device="cuda")
    pws = torch.empty(model.workspace_size(rows, L, rk.RK_WS_CLEAN_STATE | rk.RK_FLAG_CACHED_WINDOW),
                      dtype=torch.uint8, device="cuda")
    model.sensitivity_profile(batch, list(range(L)), [max(w.alphas)], s_out, pws, rows, L, window_start=P,
                              flags=rk.RK_FLAG_CACHED_WINDOW)
    s_prof = s_out.cpu().numpy()[0].astype(np.float64)
    del pws
    d_all = torch.empty(L, batch.n_seqs, dtype=torch.float32, device="cuda")
    log(f"damage inputs ready in {time.perf_counter() - t0:.1f} s (prompt {P}, window {window}, b = {b})")

    def step():
        model.compression_damage_layers(batch, P, list(range(L)), pos, Hkv * b, b, state, d_all, ws,
                                        seq_stride=L * Hkv * b)
        D = d_all.mean(dim=1).cpu().numpy().astype(np.float64)     # synchronises
        return D, rk.spearman(s_prof, D)

    for _ in range(args.warmup):
        rk.timing_begin(args.family)
        step()
        rk.timing_end()
    torch.cuda.synchronize()
    launches, fam_ms = 0, 0.0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        rk.timing_begin(args.family)
        D, rho = step()
        n, ms = rk.timing_end()
        launches += n
        fam_ms += ms
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    eval_rows = sum(T - P for T in lens)
    value = eval_rows * L / (ms_per_step / 1e3)
    avg = fam_ms / max(launches, 1)
    if args.family == "lm_kl":   # the step's L passes scored over the window rows
        flops = family_flops(args.family, cfg, eval_rows * L, 1) * args.steps / max(launches, 1)
    else:   # layer l's pass runs blocks l .. L-1 over the window rows: L (L + 1) / 2 block-passes
        flops = family_flops(args.family, cfg, eval_rows * L * (L + 1) // 2, 1) * args.steps / max(launches, 1)
    achieved = flops / (avg / 1e3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": None, "kernel": args.family,
            "launches": launches, "avg_ms": round(avg, 4), "flop_per_launch": flops}
    log(f"{args.family}: {launches} launches, avg {avg:.4f} ms, {achieved:.1f} TFLOP/s; D = {D}; rho = {rho:.3f}")
    res = {
        "metric": "window token-layers/s (isolated single-layer compression damage)",
        "value": round(value, 1), "unit": "token-layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (random-init N(0,0.02) weights, Zipf(1.1) tokens)",
        "config": {"workload": f"{w.name} compression damage: {L}L d{cfg.d_model} {cfg.n_heads}x{dh}; "
                               f"{batch.n_seqs}x{max(lens)} tokens, prompt {P} + window {window}; SnapKV b = {b} "
                               f"(window {DMG_OBS}, max pooling 7) at one layer at a time, all layers in one call",
                   "spearman_rho": None if np.isnan(rho) else round(float(rho), 4)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_damage(w, W, toks, P, b)
    print(json.dumps(res), flush=True)


def budget_tref(w) -> int:
    """Reference length of the global budget B = rho * T_ref * |A|: the common
    length of fixed-length workloads, 8192 for the variable-length set."""
    lens = w.lengths()
    return lens[0] if len(set(lens)) == 1 else 8192


def describe_lengths(lens) -> str:
    if len(set(lens)) == 1:
        return f"{len(lens)}x{lens[0]} tokens"
    return f"{len(lens)} sequences of {min(lens)}-{max(lens)} tokens (sum {sum(lens)})"


PAIR_FAMILIES = ("attention", "gemm_gate_up")


def family_step_flops(fam: str, cfg, lens, n_block_runs: int) -> float:
    """Algorithmic flops of one kernel family over `n_block_runs` block
    evaluations of a batch with sequence lengths `lens` (every row evaluated)."""
    H, dh, d, ff = cfg.n_heads, cfg.head_dim, cfg.d_model, cfg.d_ff
    if fam == "attention":
        per = sum(4.0 * H * dh * T * (T + 1) / 2 for T in lens)
    elif fam == "gemm_gate_up":
        per = 2.0 * sum(lens) * d * 2 * ff
    else:
        raise ValueError(fam)
    return per * n_block_runs


def pair_main(args):
    """Long-context profile, one step per (sequence, alpha) pair.

    A step is the whole profiling path for one calibration sequence at one
    perturbation strength: its clean reference pass (every layer, clean
    log-sum-exp), the resumed perturbed pass of every layer (prefix reuse), the
    fused LM-head + KL, the window mean, then the budget mapping of the running
    calibration mean of that alpha for every ratio and global budget.  Steps
    cycle over the pairs (sequence-major within an alpha); the whole workload is
    one cycle, whose clean passes the steps repeat once per alpha."""
    import torch
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens, upload_weights

    w = F.get_workload(args.workload)
    cfg = w.model
    t0 = time.perf_counter()
    W = F.make_weights(cfg)
    model = rk.Model(cfg, upload_weights(W))
    toks = F.make_tokens(w)
    lens = w.lengths()
    N, L = len(lens), cfg.n_layers
    alphas = list(w.alphas)
    batches = [batch_from_tokens([toks[i]], seq_index0=i) for i in range(N)]
    pairs = [(i, a) for a in range(len(alphas)) for i in range(N)]
    max_rows = max(lens)
    G = min(args.max_group, rk.RK_MAX_GROUP)
    layers = list(range(L))
    flags = 0   # eager launches: consecutive steps differ in their arguments, and ms-long kernels hide launches
    ws = torch.empty(model.workspace_size(max_rows, G, rk.RK_WS_CLEAN_STATE), dtype=torch.uint8, device="cuda")
    s_out = torch.empty(1, L, dtype=torch.float32, device="cuda")
    d_out = torch.empty(1, 1, L, dtype=torch.float32, device="cuda")
    T_ref = budget_tref(w)
    budgets = [int(round(rho * T_ref * L)) for rho in (0.1, 0.2, 0.3)]
    dsum = np.zeros((len(alphas), N, L))
    have = np.zeros((len(alphas), N), dtype=bool)
    log(f"fixtures ready in {time.perf_counter() - t0:.1f} s; {len(pairs)} (sequence, alpha) pairs, "
        f"max_rows {max_rows}, group {G}")

    def step(k):
        i, a = pairs[k % len(pairs)]
        model.sensitivity_profile(batches[i], layers, [alphas[a]], s_out, ws, max_rows, G, d_out=d_out, flags=flags)
        dsum[a, i] = d_out.cpu().numpy().astype(np.float64)[0, 0]     # synchronises
        have[a, i] = True
        s_cal = dsum[a][have[a]].mean(axis=0)        # calibration mean over the sequences done so far
        return [rk.layer_budgets(s_cal, B, r)[1] for r in w.ratios for B in budgets]

    for k in range(args.warmup):
        tw = time.perf_counter()
        rk.timing_begin(PAIR_FAMILIES[k % 2])
        step(k)
        rk.timing_end()
        log(f"warm-up step {k + 1}/{args.warmup} (pair {pairs[k % len(pairs)]}): {time.perf_counter() - tw:.2f} s")
    torch.cuda.synchronize()
    fam_ms = {f: 0.0 for f in PAIR_FAMILIES}
    fam_n = {f: 0 for f in PAIR_FAMILIES}
    fam_steps = {f: 0 for f in PAIR_FAMILIES}
    tl = 0
    t0 = time.perf_counter()
    for k in range(args.steps):
        kk = args.warmup + k
        f = PAIR_FAMILIES[k % 2]           # the timed family alternates step by step
        rk.timing_begin(f)
        step(kk)
        n, ms = rk.timing_end()
        fam_n[f] += n
        fam_ms[f] += ms
        fam_steps[f] += 1
        tl += lens[pairs[kk % len(pairs)][0]] * L
        log(f"timed step {k + 1}/{args.steps} (pair {pairs[kk % len(pairs)]}) done at "
            f"{time.perf_counter() - t0:.2f} s")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    value = tl / elapsed

    # per family: algorithmic flops per launch (block evaluations per step: the
    # clean pass's L plus sum_l (L - l) resumed ones), live HIP-event durations
    runs = L + sum(L - l for l in layers)
    kern = {}
    for f in PAIR_FAMILIES:
        if not fam_n[f]:
            continue
        per_launch = family_step_flops(f, cfg, [lens[0]], runs) / (fam_n[f] / fam_steps[f])
        avg = fam_ms[f] / fam_n[f]
        kern[f] = {"launches": fam_n[f], "avg_ms": round(avg, 4), "flop_per_launch": per_launch,
                   "achieved": round(per_launch / (avg / 1e3) / 1e12, 2),
                   "ms_per_step": round(fam_ms[f] / fam_steps[f], 1)}
    dom = max(kern, key=lambda f: kern[f]["ms_per_step"])
    kd = kern[dom]
    roof = {"bound": "mfma", "achieved": kd["achieved"], "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(kd["achieved"] / BF16_PEAK_TFLOPS, 4), "traffic": traffic_of(dom, w.name), "kernel": dom,
            "launches": kd["launches"], "avg_ms": kd["avg_ms"], "flop_per_launch": kd["flop_per_launch"]}
    for f, r in kern.items():
        log(f"{f}: {r['launches']} launches, avg {r['avg_ms']:.4f} ms, {r['achieved']:.1f} TFLOP/s, "
            f"{r['ms_per_step']:.0f} ms per step")
    pair_flops = step_flops(cfg, [lens[0]], layers, [alphas[0]])
    cfg_flops = step_flops(cfg, lens, layers, alphas)
    util = {"step_tflop": round(pair_flops / 1e12, 2), "achieved": round(pair_flops / (ms_per_step / 1e3) / 1e12, 1),
            "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(pair_flops / (ms_per_step / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
    # the whole workload (one clean pass per sequence, shared by the alphas) at the
    # steps' algorithmic rate
    wall_est = cfg_flops / (pair_flops / (ms_per_step / 1e3)) * 1e3
    res = {
        "metric": "perturbed token-layers/s (sensitivity-profile throughput)",
        "value": round(value, 1), "unit": "token-layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (random-init N(0,0.02) weights, Zipf(1.1) tokens)",
        "launch": "eager",
        "config": {"workload": f"{w.name}: {L}L d{cfg.d_model} {cfg.n_heads}q/{cfg.n_kv_heads}kv x{cfg.head_dim} "
                               f"FFN{cfg.d_ff} V{cfg.vocab} theta {cfg.rope_theta:g}; {describe_lengths(lens)}; "
                               f"alpha {alphas}; all layers; ratios {list(w.ratios)}; budgets {budgets}; one step = "
                               f"one (sequence, alpha) pair: its clean pass, all {L} perturbed passes, fused "
                               f"LM-head + KL, means and the budget mapping; steps cycle over the {len(pairs)} pairs",
                   "perturbed_token_layers_per_step": lens[0] * L,
                   "profile_wall_ms_est": round(wall_est, 1),
                   "profile_wall_note": "whole workload (one clean pass per sequence) at the steps' algorithmic "
                                        f"rate: {cfg_flops / 1e15:.2f} PFLOP"},
        "roofline": roof,
        "kernels": kern,
        "mfma_util": util,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, W, toks)
    print(json.dumps(res), flush=True)


def fp32_cost_main(args):
    """Cost of the fp32 path (every operand and activation fp32, the bf16 weights
    upcast exactly) against the bf16 path on the same model: the profile of the
    first `--fp32-tokens` tokens of sequence 0 at the last and the middle layer
    (largest alpha), timed with each dtype.  The fp32 path is the option that
    meets the 1e-4 fp32 logit bar at 32 layers; this prices it."""
    import dataclasses
    import torch
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens, upload_weights

    w = F.get_workload(args.workload)
    cfg16 = w.model
    T = int(args.fp32_tokens)
    toks = [F.make_tokens(w)[0][:T]]
    layers = [cfg16.n_layers - 1, cfg16.n_layers // 2]
    alpha = max(w.alphas)
    W16 = F.make_weights(cfg16)
    out = {}
    for name, cfg, W in (("bf16", cfg16, W16),
                         ("f32", dataclasses.replace(cfg16, dtype="f32"), F.f32_weights(cfg16, W16))):
        model = rk.Model(cfg, upload_weights(W))
        batch = batch_from_tokens(toks)
        wsf = rk.RK_WS_CLEAN_STATE | (rk.RK_FLAG_UNFUSED_KL if name == "f32" else 0)
        ws = torch.empty(model.workspace_size(batch.rows, len(layers), wsf), dtype=torch.uint8, device="cuda")
        s_out = torch.empty(1, len(layers), dtype=torch.float32, device="cuda")
        run = lambda: model.sensitivity_profile(batch, layers, [alpha], s_out, ws, batch.rows, len(layers))
        run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            run()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        fl = step_flops(cfg16, [T], layers, [alpha])
        out[name] = {"ms_per_profile": round(ms, 2), "tflop_per_s": round(fl / (ms / 1e3) / 1e12, 2),
                     "s": [float(x) for x in s_out.cpu().numpy()[0]]}
        log(f"{name}: {ms:.1f} ms per profile, {fl / (ms / 1e3) / 1e12:.1f} TFLOP/s")
        del model, ws, s_out
        torch.cuda.empty_cache()
    res = {"metric": "fp32-path cost (profile wall time, fp32 vs bf16)", "workload":
           f"{w.name}: first {T} tokens of sequence 0, layers {layers}, alpha {alpha}",
           "bf16": out["bf16"], "f32": out["f32"],
           "f32_over_bf16": round(out["f32"]["ms_per_profile"] / out["bf16"]["ms_per_profile"], 1)}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b-long-bf16")
    ap.add_argument("--step-unit", choices=("auto", "pair", "profile"), default="auto",
                    help="pair: one step = one (sequence, alpha) pair of the profile; profile: one step = the "
                         "whole profile of the workload; auto: pair for the 2x32768 workload, else profile")
    ap.add_argument("--max-group", type=int, default=12)
    ap.add_argument("--join", type=int, default=0,
                    help="whole-profile steps: max_rows = JOIN x the batch rows, so up to JOIN resumed passes of a "
                         "group run layer-synchronously (0: 4 for batches of at most 16384 rows, else 1)")
    ap.add_argument("--family", default="gemm_gate_up", help="kernel family for the roofline figure")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying a HIP graph")
    ap.add_argument("--signal", choices=("downstream", "local"), default="downstream",
                    help="profile signal: the KL of the final distributions (the method) or the layer-local "
                         "response of the perturbed block (the w/o DS ablation)")
    ap.add_argument("--fp32-cost", action="store_true",
                    help="price the fp32 path against the bf16 path on a prefix of the workload's first sequence")
    ap.add_argument("--fp32-tokens", type=int, default=2048)
    ap.add_argument("--unfused-kl", action="store_true",
                    help="score the passes through materialised fp32 logits and the separate KL kernel "
                         "(the verification path) instead of the fused LM-head + KL")
    ap.add_argument("--window", type=int, default=0,
                    help="cached-window mode: evaluate the last WINDOW tokens of every sequence against the cached "
                         "prefix (0: the resumed full-sequence profile)")
    ap.add_argument("--snapkv", action="store_true",
                    help="time the SnapKV selection with per-layer budgets (the budgets' consumer) instead")
    ap.add_argument("--policy", action="store_true",
                    help="the damage of whole per-layer budget policies (RippleKV vs uniform) in the cached-window "
                         "split, every layer compressed at once")
    ap.add_argument("--damage", action="store_true",
                    help="time the isolated single-layer compression damage of every layer instead (prompt = all "
                         "but the last WINDOW tokens, default 256)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (calibrates HBM byte counters)")
    ap.add_argument("--derive-traffic", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="print the per-launch HBM bytes of --family from rocprofv3 --pmc csv directories")
    ap.add_argument("--derive-traffic-table", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="print HBM bytes and GB/s of every kernel family from the same four directories")
    ap.add_argument("--derive-counters", nargs="+", metavar="DIR",
                    help="print MFMA-busy, waiting and clock figures per kernel family from rocprofv3 --pmc "
                         "csv directories")
    args = ap.parse_args()
    if args.derive_traffic:
        print(json.dumps(derive_traffic(*args.derive_traffic, args.family)))
        return
    if args.derive_traffic_table:
        derive_traffic_table(*args.derive_traffic_table)
        return
    if args.derive_counters:
        derive_counters(args.derive_counters)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the profile's passes are independent and "
              "would shard by sequence or layer, which is not implemented", file=sys.stderr)
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
    if args.fp32_cost:
        fp32_cost_main(args)
        return
    if args.snapkv:
        snapkv_main(args)
        return
    if args.damage:
        damage_main(args)
        return
    if args.policy:
        policy_main(args)
        return
    unit = args.step_unit
    if unit == "auto":
        unit = "pair" if args.workload == "llama3-8b-long-bf16" and args.window == 0 and args.signal == "downstream" \
            else "profile"
    if unit == "pair":
        if args.window or args.signal != "downstream":
            raise SystemExit("--step-unit pair runs the resumed downstream profile only")
        pair_main(args)
        return
    import fixtures as F
    import paper_2608_08684_amd as rk
    from paper_2608_08684_amd.inputs import batch_from_tokens as make_batch, upload_weights

    w = F.get_workload(args.workload)
    cfg = w.model
    t0 = time.perf_counter()
    W = F.make_weights(cfg)
    dw = upload_weights(W)
    toks = F.make_tokens(w)
    batch = make_batch(toks)
    model = rk.Model(cfg, dw)
    log(f"fixtures ready in {time.perf_counter() - t0:.1f} s")

    layers = list(range(cfg.n_layers))
    alphas = list(w.alphas)
    rows = batch.rows
    G = min(args.max_group, rk.RK_MAX_GROUP)
    window = int(args.window)
    local = args.signal == "local"
    flags = ((rk.RK_FLAG_CACHED_WINDOW if window > 0 else 0) | (0 if args.no_graph else rk.RK_FLAG_GRAPH) |
             (rk.RK_FLAG_LOCAL_SIGNAL if local else 0) | (rk.RK_FLAG_UNFUSED_KL if args.unfused_kl else 0))
    P = min(w.lengths()) - window if window > 0 else 0
    if window > 0 and P < 1:
        raise SystemExit(f"--window {window} leaves no prefix in the shortest sequence")
    # default: up to 4 resumed passes per launch for batches of at most 16384 rows
    join = args.join if args.join > 0 else (4 if rows <= 16384 else 1)
    max_rows = join * rows
    ws = torch.empty(model.workspace_size(max_rows, G, rk.RK_WS_CLEAN_STATE |
                                          (flags & (rk.RK_FLAG_CACHED_WINDOW | rk.RK_FLAG_LOCAL_SIGNAL |
                                                    rk.RK_FLAG_UNFUSED_KL))),
                     dtype=torch.uint8, device="cuda")
    s_out = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
    d_out = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda")
    T_ref = budget_tref(w)
    budgets = [int(round(rho * T_ref * len(layers))) for rho in (0.1, 0.2, 0.3)]

    def step():
        model.sensitivity_profile(batch, layers, alphas, s_out, ws, max_rows, G, d_out=d_out, window_start=P,
                                  flags=flags)
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
    for k in range(args.warmup):
        tw = time.perf_counter()
        rk.timing_begin(args.family)
        step()
        rk.timing_end()
        log(f"warm-up step {k + 1}/{args.warmup}: {time.perf_counter() - tw:.2f} s")
    torch.cuda.synchronize()
    launches, fam_ms = 0, 0.0
    t0 = time.perf_counter()
    for k in range(args.steps):
        rk.timing_begin(args.family)
        step()
        n, ms = rk.timing_end()
        launches += n
        fam_ms += ms
        if args.steps <= 3 or k + 1 == args.steps:
            log(f"timed step {k + 1}/{args.steps} done at {time.perf_counter() - t0:.2f} s")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    eval_rows = sum(T - P for T in w.lengths())     # rows each pass recomputes (all rows unless cached window)
    tokens_layers = eval_rows * len(layers) * len(alphas)
    value = tokens_layers / (ms_per_step / 1e3)

    fam_avg_ms = fam_ms / max(launches, 1)
    hbm_family = args.family == "kl_logits"
    if hbm_family:
        # one launch scores a group of passes: every logit of the clean rows and of
        # each pass read once, one fp32 KL per row and pass written
        n_launch_pass = len(layers) * len(alphas) / max(launches / args.steps, 1)
        flops = (1 + n_launch_pass) * eval_rows * cfg.vocab * 4.0 + n_launch_pass * eval_rows * 4.0
    elif args.family == "lm_kl":
        n_pass_lm = G  # perturbed passes scored per LM-head launch (algorithmic: pert logits only)
        flops = family_flops(args.family, cfg, eval_rows, n_pass_lm)
    else:
        # a projection family's rows over the step: the reference pass (the prefix
        # prefill and the window in the cached-window mode) and every resumed layer
        # of every pass; in the cached-window mode one launch carries the window
        # rows of several passes, so the flops per launch are the step's over its
        # launches
        L = cfg.n_layers
        pass_layers = sum(L - l for l in layers) * len(alphas)
        rows_total = rows * L + eval_rows * pass_layers if window == 0 else \
            (rows - eval_rows) * L + eval_rows * L + eval_rows * pass_layers
        flops = family_flops(args.family, cfg, rows_total, 1) * args.steps / max(launches, 1)
    achieved = flops / (fam_avg_ms / 1e3) / (1e9 if hbm_family else 1e12)
    traffic = traffic_of(args.family, w.name, min(join, G, 64 // batch.n_seqs) if window == 0 and not local else 1)
    if hbm_family:
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": args.family,
                "launches": launches, "avg_ms": round(fam_avg_ms, 4), "bytes_per_launch": flops}
    else:
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": args.family, "launches": launches, "avg_ms": round(fam_avg_ms, 4),
                "flop_per_launch": flops}
    log(f"{args.family}: {launches} launches, avg {fam_avg_ms:.4f} ms, {achieved:.1f} "
        f"{'GB/s' if hbm_family else 'TFLOP/s'}")
    # the whole step's MFMA utilisation: its algorithmic work over the step time
    sf = step_flops(cfg, w.lengths(), layers, alphas, P, local)
    util = {"step_tflop": round(sf / 1e12, 2), "achieved": round(sf / (ms_per_step / 1e3) / 1e12, 1),
            "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(sf / (ms_per_step / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4)}

    mode = "" if window == 0 else f"; cached window: prefix {P}, window {window} per sequence"
    mode += "; layer-local signal (w/o DS ablation)" if local else ""
    mode += "; unfused KL (materialised fp32 logits, separate KL kernel)" if args.unfused_kl else ""
    metric = ("perturbed token-layers/s (sensitivity-profile throughput)" if window == 0 else
              "perturbed window token-layers/s (cached-window sensitivity-profile throughput)")
    if local:
        metric = metric.replace("sensitivity-profile", "layer-local-signal profile")
    res = {
        "metric": metric,
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
                               f"FFN{cfg.d_ff} V{cfg.vocab}; {describe_lengths(w.lengths())}; "
                               f"alpha {alphas}; all layers; ratios {list(w.ratios)}; budgets {budgets}{mode}",
                   "perturbed_token_layers_per_step": tokens_layers, "profile_wall_ms": round(ms_per_step, 3),
                   "passes_per_launch": min(join, G, 64 // batch.n_seqs) if window == 0 and not local else 1},
        "roofline": roof,
        "mfma_util": util,
    }
    if not args.no_cpu_baseline:
        if window == 0:
            res["cpu_baseline"] = cpu_baseline(w, W, toks, local=local)
        elif not local:
            res["cpu_baseline"] = cpu_baseline_window(w, W, toks, window)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
