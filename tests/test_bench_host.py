"""Host-side accounting of bench.py (no GPU): the exact causal flop count and
the argument contract for several GPUs."""

from __future__ import annotations

import subprocess
import sys
from pathlib import Path

import numpy as np

import bench
from synth import WORKLOADS

ROOT = Path(__file__).resolve().parents[1]


def test_exact_causal_flops_of_full_lists_is_the_dense_causal_count():
    # Every block 0..i in every row: the pairs (query, key <= query) of dense
    # causal attention, N (N + 1) / 2 per head, 4 d flops each (QK^T and PV).
    for n in (2048, 2000, 64, 1):
        w = WORKLOADS["tiny-2k"].with_(seq_len=n)
        counts = np.tile(np.arange(1, w.n_blocks + 1), (w.n_q_heads, 1))
        assert bench.exact_causal_flops(w, counts) == 4 * w.head_dim * w.n_q_heads * n * (n + 1) // 2


def test_exact_causal_flops_of_diagonal_only_lists():
    # Only the diagonal block of each row: B (B + 1) / 2 pairs per full block.
    w = WORKLOADS["tiny-2k"]
    B = w.block_size
    counts = np.ones((w.n_q_heads, w.n_blocks), dtype=np.int64)
    assert bench.exact_causal_flops(w, counts) == 4 * w.head_dim * w.n_q_heads * w.n_blocks * B * (B + 1) // 2


def test_algorithmic_attention_flops_count_whole_blocks():
    w = WORKLOADS["tiny-2k"]
    alg = bench.algorithmic(w, 10)
    assert alg["attn_flops"] == 4 * w.block_size ** 2 * w.head_dim * 10
    assert alg["pairs"] == w.n_q_heads * w.n_blocks * (w.n_blocks + 1) // 2


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr)


def test_cpu_baseline_covers_every_kv_head_and_states_its_sample():
    """The CPU oracle timing: statistics of all KV heads in full, the stated
    row samples, the cores this process may use, and the CPU model."""
    import os
    import oracle
    from synth import f64_from_bf16_bits, make_inputs
    w = WORKLOADS["tiny-2k"].with_(seq_len=512)
    inp = make_inputs(w)
    C, R = oracle.block_stats(f64_from_bf16_bits(inp["k"]), w.block_size)
    M = w.n_blocks
    counts = np.tile(np.arange(1, M + 1, dtype=np.int32), (w.n_q_heads, 1))
    indices = np.zeros((w.n_q_heads, M * (M + 1) // 2), dtype=np.int32)
    for i in range(M):
        indices[:, i * (i + 1) // 2:i * (i + 1) // 2 + i + 1] = np.arange(i + 1)
    cb = bench.cpu_baseline(w, inp, counts, indices, 4, 2)
    assert cb["cores"] == len(os.sched_getaffinity(0))
    assert cb["kind"] == "oracle" and cb["unit"] == "ms/layer" and cb["value"] > 0
    assert f"all {w.n_kv_heads} KV heads in full" in cb["sample"]
    assert "selection for 4" in cb["sample"] and "attention (on the GPU's lists) for 2" in cb["sample"]
    assert cb["cpu"]


def test_density_context_starts_with_the_workloads_thresholds():
    """The threshold sweep repeats the headline pair first (its attention time
    calibrates the others), holds the paper's default pair, and keeps every
    pair inside [0, 1]."""
    w = WORKLOADS["qwen3-30b-a3b-128k"]
    assert bench.TAU_SWEEP[0] == (w.tau_base, w.tau_rescue)
    assert (0.22, 0.18) in bench.TAU_SWEEP
    assert all(0.0 <= t <= 1.0 for pair in bench.TAU_SWEEP for t in pair)


def test_unit_rate_summary_reads_the_probe_cases(monkeypatch, tmp_path):
    """The brief unit-rate summary picks the right cases out of the probe's
    JSON: per-instruction cycles at two waves per SIMD, the dependent chain at
    one wave, and the LDS read rates (4 SIMDs x 2 waves x 16 reads per
    iteration)."""
    import json

    def case(other, n, w, cyc, mf=0, chains=4):
        return {"mfma": mf, "acc": "vgpr", "acc_chains": chains, "other": other, "n_other": n,
                "placement": "same_wave", "waves_per_simd": w, "cycles_per_iter_mfma_wave": cyc,
                "cycles_per_iter_other_wave": 0.0, "sclk_mhz": 2000, "ms": 1.0, "simd_of_wave": []}
    data = {"cases": [case("v_exp_f32", 8, 2, 152.0), case("v_fma_f32", 8, 2, 64.0),
                      case("none", 0, 2, 512.0, mf=8), case("none", 0, 1, 256.0, mf=8, chains=1),
                      case("none", 0, 1, 999.0, mf=8), case("softmax_mix", 28, 2, 760.0, mf=8),
                      case("ds_read_b128", 16, 2, 512.0), case("ds_read_b64_tr_b16", 16, 2, 256.0)],
            "attention_block_loop": [{"schedule": "free_running", "mfma_busy": 0.75}]}
    probe = tmp_path / "probe"
    probe.write_text("#!/bin/sh\ncat <<'JSON'\n" + json.dumps(data) + "\nJSON\n")
    probe.chmod(0o755)
    monkeypatch.setattr(bench, "UNIT_RATES_BIN", str(probe))
    r = bench.unit_rates(brief=True)
    assert r["exp_cycles"] == 9.5 and r["fma_cycles"] == 4.0 and r["mfma_32x32x16_bf16_cycles"] == 32.0
    assert r["mfma_cycles_dependent_chain"] == 32.0
    assert r["mfma_cycles_with_softmax_mix"] == 47.5
    assert r["lds_read_bytes_per_clk_per_cu"] == {"ds_read_b128": 256.0, "ds_read_b64_tr_b16": 256.0}
    assert r["block_loop_mfma_busy"] == {"free_running": 0.75}
