"""The sensitivity profile driven from plain C (tests/c/abi_gpu.c): device memory
from the HIP runtime, no Python or torch in the process.  The same model, batch
and arguments through the ctypes binding give bitwise the same profile s and
the same budgets.  (The driver is built with the host C compiler, a second.)"""
import os
import shutil
import struct
import subprocess

import numpy as np
import pytest

import fixtures as F

from gpu_helpers import Runner, log, make_batch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CASES = [
    F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                  rope_theta=1.0e4, dtype="bf16"),
    F.small_model(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32, d_ff=256, vocab=512,
                  rope_theta=1.0e4, dtype="f32"),
]


def _build(tmp):
    import paper_2608_08684_amd as rk
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = os.path.join(tmp, "abi_gpu")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-isystem", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_gpu.c"), rk.LIB_PATH,
                    "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + os.path.join(rocm, "lib") + ":" + os.path.dirname(rk.LIB_PATH), "-o", exe],
                   check=True)
    return exe


def _write(path, cfg, W, toks, alphas):
    offs = np.concatenate([[0], np.cumsum([len(t) for t in toks])]).astype(np.int64)
    dt = 1 if cfg.dtype == "bf16" else 0

    def mat(a):
        return np.ascontiguousarray(a).tobytes()   # bf16 bit patterns or fp32, as on the device

    def vec(a):
        return np.ascontiguousarray(a, dtype=np.float32).tobytes()
    with open(path, "wb") as f:
        f.write(struct.pack("<10i", cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff,
                            cfg.vocab, dt, len(toks), len(alphas)))
        f.write(struct.pack("<2f", cfg.rope_theta, cfg.rms_eps))
        f.write(offs.tobytes())
        f.write(np.asarray(alphas, dtype=np.float32).tobytes())
        f.write(mat(W["tok_emb"]))
        for l in range(cfg.n_layers):
            f.write(mat(W["w_qkv"][l]) + mat(W["w_o"][l]) + mat(W["w_gate_up"][l]) + mat(W["w_down"][l]))
            f.write(vec(W["attn_norm"][l]) + vec(W["mlp_norm"][l]))
        f.write(vec(W["final_norm"]) + mat(W["lm_head"]))
        f.write(np.concatenate(toks).astype(np.int32).tobytes())


@pytest.mark.parametrize("case", range(len(CASES)))
def test_profile_from_c_equals_the_binding(case, tmp_path):
    import paper_2608_08684_amd as rk
    cfg = CASES[case]
    exe = _build(str(tmp_path))
    W = F.make_weights(cfg)
    toks = F.make_tokens(F.make_workload("cabi", cfg, [200, 77], seed_id=97 + case))
    alphas = [0.05, 0.1]
    data = str(tmp_path / "in.bin")
    _write(data, cfg, W, toks, alphas)
    log(f"case {case}: running the C driver")
    out = subprocess.run([exe, data], check=True, capture_output=True, text=True, timeout=120).stdout
    got = {line.split()[0]: line.split()[1:] for line in out.splitlines()}
    run = Runner(cfg, W)
    batch = make_batch(toks)
    L = cfg.n_layers
    s, _ = run.profile(batch, list(range(L)), alphas, max_group=L, want_d=False)
    for k in range(len(alphas)):
        c_s = np.array([float(x) for x in got[f"s{k}"]], dtype=np.float32)
        np.testing.assert_array_equal(c_s, s[k].astype(np.float32))
    _, b = rk.layer_budgets(s[-1], 100 * L, 2.0)
    assert got["budgets"][0] == "0" and [int(x) for x in got["budgets"][1:]] == list(b)
    log(f"case {case}: s from C = s from the binding: {s.tolist()}; budgets {list(b)}")
