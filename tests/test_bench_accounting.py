"""bench.py's accounting, on the CPU: the active-row counts and reuse rate it derives from a
reuse map, the algorithmic FLOPs and bytes it divides by measured times (the per-row figure of
the method: 24 D^2 for the four linear layers plus 4 N D for attention over all N keys), and its
refusal of more than one GPU."""
import os
import subprocess
import sys

import numpy as np

import bench
import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _masks(F=12, L=3, N=7, G=4, seed=0):
    rng = np.random.default_rng(seed)
    m = (rng.random((F, L, N)) < 0.6).astype(np.uint8)
    m[::G] = 0          # reference frames are never reused
    m[:, :, 0] = 0      # nor is the class token
    return m


def test_active_rows_count_every_recomputed_token_and_whole_reference_frames():
    G = 4
    m = _masks(G=G)
    F, L, N = m.shape
    want = np.zeros(L, np.int64)
    for f in range(F):
        for layer in range(L):
            for i in range(N):
                if f % G == 0 or m[f, layer, i] == 0:
                    want[layer] += 1
    assert np.array_equal(bench.active_rows(m, G), want)


def test_reuse_rate_matches_the_oracle_definition():
    for G in (2, 4, 5):
        m = _masks(F=13, G=G, seed=G)
        assert abs(bench.reuse_of(m, G) - oracle.reuse_rate(m, G)) < 1e-12


def test_linear_and_attention_flops_per_row_are_the_method_s_count():
    m = synth.get_config("vit_l14").model
    D, N = m.width, m.n_tokens
    per_row_linear = sum(bench.stage_flops(s, m, 1) for s in ("qkv", "oproj", "fc1", "fc2"))
    assert per_row_linear == 24 * D * D          # MLP width 4 D: 6 + 2 + 8 + 8 D^2
    assert bench.stage_flops("attn", m, 1) == 4 * N * D
    assert bench.stage_flops("gate", m, 1000) == 0.0
    assert bench.stage_flops("qkv", m, 10) == 10 * bench.stage_flops("qkv", m, 1)


def test_gemm_bytes_by_hand():
    m = synth.get_config("vit_b16").model        # D 768, MLP 3072
    D, Dm, M = 768, 3072, 1000
    assert (m.width, m.mlp) == (D, Dm)
    # QKV: bf16 rows in, bf16 weights, bf16 q/k/v rows out
    assert bench.stage_bytes("qkv", m, M) == M * D * 2 + 3 * D * D * 2 + M * 3 * D * 2
    # FC2: bf16 hidden rows, bf16 weights, fp32 residual rows in, row indices, fp32 rows out
    assert bench.stage_bytes("fc2", m, M) == M * Dm * 2 + D * Dm * 2 + M * D * 4 + M * 4 + M * D * 4
    # attention: packed query rows in and outputs out, and each frame's N keys and values once
    F, N = 16, m.n_tokens
    assert bench.attn_bytes(m, M, F) == M * D * 2 * 2 + F * N * 2 * D * 2
    # LN2: fp32 rows in, bf16 rows out
    assert bench.row_stage_bytes("ln2", m, 0, M, F) == M * D * 6


def test_more_than_one_gpu_is_refused_before_any_device_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
