#!/usr/bin/env python
"""Benchmark of the RBS sparse-prefill hot path on one MI355X.

One step = one pass of the whole path over one attention layer's inputs:
block statistics -> dual-branch selection -> block-sparse attention, with every
input already resident in HBM.  The default workload is the 128K
Qwen3-30B-A3B-shaped layer (32 query / 4 KV heads, d = 128, B = 128), seeded
synthetic data.  Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "128K sparse prefill-attn ms/layer, speedup vs own dense, MFMA util %"
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E, vendor figure
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA, vendor figure (no sparsity)
PROFILES = os.path.join(ROOT, "profiles")


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default=None,
                   help="workload name (default: qwen3-30b-a3b-128k; the study defaults to qwen3-30b-a3b-32k)")
    p.add_argument("--dense-reps", type=int, default=2)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--flush-gib", type=float, default=1.0,
                   help="also time the steps with a read of this many GiB of scratch between them, outside "
                        "the timed events, so that no step finds the previous one's data in L2 or the Infinity "
                        "Cache (0 skips)")
    p.add_argument("--no-tau-sweep", dest="tau_sweep", action="store_false",
                   help="skip the attention times of the same layer selected at tighter thresholds")
    p.add_argument("--no-extra-configs", action="store_true",
                   help="skip the compact lines for the other workloads (128K at B = 64 and 256, 32K, the "
                        "64-head 64K layer)")
    p.add_argument("--unit-rates", action="store_true",
                   help="instead of the benchmark line: the measured issue rates of the exponential, FMA, LDS "
                        "and matrix instructions (the unit-rate probe, built with the library)")
    p.add_argument("--cpu-select-rows", type=int, default=256,
                   help="sampled (head, query block) rows for the oracle's selection timing")
    p.add_argument("--cpu-attn-rows", type=int, default=24,
                   help="sampled (head, query block) rows for the oracle's attention timing")
    p.add_argument("--fused-steps", type=int, default=5,
                   help="also time this many steps through the fused select-then-attend entry (0 skips)")
    p.add_argument("--selector-study", action="store_true",
                   help="instead of the benchmark line: needle recall and dense-attention-mass coverage vs "
                        "density of the method and the supporting selectors (default workload: the 32K layer)")
    p.add_argument("--study-needle-norm", type=float, default=None,
                   help="norm of the planted needle keys for the study (default: the workload's, 3)")
    p.add_argument("--study-rows", type=int, default=256,
                   help="sampled (head, query block) rows for the attention-mass coverage")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a 1 GiB device copy (for scaling HBM counters)")
    p.add_argument("--batch", type=int, default=0,
                   help="instead of the benchmark line: a batch of this many independent sequences of the "
                        "workload's length through the varlen calls, against the same sequences one call "
                        "at a time and against the dense path at the same batch")
    p.add_argument("--batch-lens", default=None,
                   help="comma-separated sequence lengths for the batch mode (overrides --batch)")
    p.add_argument("--fp8", action="store_true",
                   help="instead of the benchmark line: the attention stage on FP8 (E4M3) inputs over the same "
                        "lists, against the bf16 attention and the FP8 dense path, plus the packing time")
    p.add_argument("--layer-sweep", type=int, default=0,
                   help="instead of the benchmark line: this many layers of the 128K layer schedule "
                        "(per-layer key noise and needle counts), per-layer density and times, sparse vs "
                        "dense, serial and with the next layer's stats and selection on a second stream")
    return p.parse_args()


PEAK_SCLK_MHZ = 2400.0        # clock the vendor MFMA figure assumes


class SclkSampler:
    """Shader clock while a region runs: a thread reads the current level of
    the GPU's pp_dpm_sclk (sysfs, the starred line) every 5 ms.  None when the
    file is not readable."""

    def __init__(self):
        import glob
        files = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = files[0] if len(files) == 1 else None
        self.mhz = []
        self._stop = False
        self._thread = None

    def _read(self):
        try:
            with open(self.path) as f:
                for line in f:
                    if line.rstrip().endswith("*"):
                        return float(line.split(":")[1].strip().lower().split("mhz")[0])
        except (OSError, ValueError, IndexError):
            return None
        return None

    def _run(self):
        while not self._stop:
            v = self._read()
            if v is not None:
                self.mhz.append(v)
            time.sleep(0.005)

    def __enter__(self):
        if self.path is not None:
            import threading
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop = True
        if self._thread is not None:
            self._thread.join()

    def summary(self):
        import numpy as np
        if not self.mhz:
            return None
        a = np.array(self.mhz)
        return {"median": float(np.median(a)), "min": float(a.min()), "max": float(a.max()), "samples": len(a),
                "source": self.path}


def copy_ceiling_gbps(torch, dev, reps: int = 5) -> float:
    """Device-to-device copy of 1 GiB (read + write counted), median of reps."""
    import numpy as np
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    del src, dst
    return 2.0 * (1 << 30) / (float(np.median(ts)) * 1e-3) / 1e9


def exact_causal_flops(w, counts_np) -> int:
    """QK^T and PV flops over the (query, key) pairs with key <= query of the
    executed blocks: full B x B blocks off the diagonal (every list holds the
    diagonal block, and only the last key block can be partial, which only a
    diagonal can be), nq (nq + 1) / 2 pairs on it."""
    import numpy as np
    N, B, d, M = w.seq_len, w.block_size, w.head_dim, w.n_blocks
    nq = np.minimum(B, N - np.arange(M) * B).astype(np.int64)
    per_row = (counts_np.astype(np.int64) - 1) * nq[None, :] * B + (nq * (nq + 1) // 2)[None, :]
    return int(4 * d * per_row.sum())


def algorithmic(w, counts_sum: int):
    """Bytes / flops each stage must move or compute per launch."""
    N, Hq, Hkv, d, B = w.seq_len, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size
    M = w.n_blocks
    pairs = Hq * M * (M + 1) // 2
    stats_bytes = Hkv * N * d * 2 + Hkv * M * d * 4 + Hkv * M * d * 2 + Hkv * M * 4 * 3 + Hkv * 8
    select_bytes = Hq * N * d * 2 + Hkv * M * (d * 2 + 4) + Hq * M * 4 + counts_sum * 4
    select_flops = 2 * B * d * pairs            # q . c_b for every causal (token, block) pair
    attn_flops = 4 * B * B * d * counts_sum     # QK^T and PV over every executed block pair
    dense_flops = 4 * B * B * d * pairs
    return dict(stats_bytes=stats_bytes, select_bytes=select_bytes, select_flops=select_flops,
                attn_flops=attn_flops, dense_flops=dense_flops, pairs=pairs)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, inp, counts_np, indices_np, n_select: int, n_attn: int):
    """Time the float64 oracle on the host cores, on a bounded sample of the
    same workload, scaled to one layer (ms/layer): block statistics and radius
    quantiles over every KV head in full; selection and attention (on the GPU's
    lists) on random (query head, query block) rows, each scaled to all rows.
    NumPy's BLAS threads are set to the cores this process may run on."""
    import numpy as np
    import oracle
    from synth import f64_from_bf16_bits
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # pragma: no cover
        limiter = None
    M, B, G = w.n_blocks, w.block_size, w.group
    rng = np.random.default_rng(123)
    rows = [(int(rng.integers(w.n_q_heads)), int(rng.integers(M))) for _ in range(max(n_select, n_attn))]

    t0 = time.perf_counter()
    Kf = f64_from_bf16_bits(inp["k"])
    C, R = oracle.block_stats(Kf, B)
    beta, _ = oracle.rescue_coefficients(R)
    t_stats = time.perf_counter() - t0

    Vf = f64_from_bf16_bits(inp["v"])
    t_sel = 0.0
    t_att = 0.0
    for k, (h, i) in enumerate(rows):
        s, e = i * B, min((i + 1) * B, w.seq_len)
        qi = f64_from_bf16_bits(inp["q"][h, s:e])
        if k < n_select:
            t0 = time.perf_counter()
            oracle.select_row(qi, C[h // G], R[h // G], beta[h // G], i, M, w.tau_base, w.tau_rescue,
                              w.n_sink, w.n_local, w.n_recent)
            t_sel += time.perf_counter() - t0
        if k >= n_attn:
            continue
        base = i * (i + 1) // 2
        ids = indices_np[h, base:base + counts_np[h, i]].tolist()
        qh = np.zeros((e, w.head_dim))
        qh[s:e] = qi
        t0 = time.perf_counter()
        oracle.attention_rows(qh, Kf[h // G], Vf[h // G], B, i, ids)
        t_att += time.perf_counter() - t0
    if limiter is not None:
        limiter.unregister()
    total_rows = w.n_q_heads * M
    ms = (t_stats + t_sel / n_select * total_rows + t_att / n_attn * total_rows) * 1e3
    return {"value": ms, "unit": "ms/layer", "cores": int(cores), "kind": "oracle", "cpu": _cpu_model(),
            "sample": (f"float64 numpy oracle on {cores} host cores: block statistics and radius quantiles of "
                       f"all {w.n_kv_heads} KV heads in full ({t_stats:.2f} s); selection for {n_select} and "
                       f"attention (on the GPU's lists) for {n_attn} random (query head, query block) rows of "
                       f"{total_rows}, each scaled to all rows ({t_sel:.2f} s, {t_att:.2f} s measured)"),
            "measured_s": t_stats + t_sel + t_att}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the RBS hot path is built and "
                                   "measured per GPU (heads would shard across GPUs with no communication)",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_20971_amd as rbs
    from synth import workload, make_inputs

    if args.selector_study:
        return selector_study(args)
    if args.batch or args.batch_lens:
        return batch_bench(args)
    if args.layer_sweep:
        return layer_sweep(args)
    if args.fp8:
        return fp8_bench(args)
    if args.unit_rates:
        print(json.dumps(unit_rates()), flush=True)
        return
    w = workload(args.workload or "qwen3-30b-a3b-128k")
    _log(f"[bench] workload {w.name}: N={w.seq_len} Hq={w.n_q_heads} Hkv={w.n_kv_heads} B={w.block_size}")
    t0 = time.perf_counter()
    inp = make_inputs(w)
    _log(f"[bench] inputs generated in {time.perf_counter() - t0:.1f}s")

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    Q, K, V = up(inp["q"]), up(inp["k"]), up(inp["v"])
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    stats = rbs.BlockStats.allocate(shape, dev)
    counts, indices = rbs.allocate_lists(shape, dev)
    O = torch.empty_like(Q)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        rbs.rbs_block_stats(shape, K, stats, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        rbs.rbs_select(shape, Q, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent,
                       counts, indices, stream=stream)
        if ev is not None:
            ev[2].record(stream)
        rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, O, stream=stream)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    _log(f"[bench] warmup done ({args.warmup} steps)")

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    with SclkSampler() as sclk:
        t_start = time.perf_counter()
        for k in range(args.steps):
            step(events[k])
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t_start) * 1e3 / args.steps
    per_step = np.array([[ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]), ev[2].elapsed_time(ev[3])]
                         for ev in events])
    stage_ms = per_step.mean(axis=0)
    # Medians beside the means: the first timed step starts on an idle GPU
    # (the loop begins after a synchronize), so its first stage also holds the
    # host's time to issue it; the later steps are queued behind the previous
    # step's attention.
    stage_med = np.median(per_step, axis=0)
    ms_per_step = float(stage_ms.sum())
    _log(f"[bench] timed {args.steps} steps: stats {stage_ms[0]:.3f} ms, select {stage_ms[1]:.3f} ms, "
         f"attention {stage_ms[2]:.3f} ms (wall {wall_ms:.3f} ms/step)")

    # The same steps with the caches flushed between them, outside the events:
    # a read of a scratch buffer larger than L2 plus the 256 MiB Infinity
    # Cache.  A read leaves clean lines behind; a write would leave the cache
    # full of dirty ones, whose write-back the next step's reads would pay for.
    flushed = None
    if args.flush_gib > 0:
        scratch = torch.ones(int(args.flush_gib * (1 << 28)), dtype=torch.float32, device=dev)
        fev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        sink = torch.zeros((), dtype=torch.float32, device=dev)
        for k in range(args.steps):
            torch.sum(scratch, dim=0, out=sink)
            step(fev[k])
        torch.cuda.synchronize()
        del sink
        fms = np.zeros(3)
        for ev in fev:
            fms += [ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]), ev[2].elapsed_time(ev[3])]
        fms /= args.steps
        del scratch
        flushed = {"flush_gib": args.flush_gib, "ms_per_step": round(float(fms.sum()), 4),
                   "stats_ms": round(float(fms[0]), 4), "select_ms": round(float(fms[1]), 4),
                   "attn_ms": round(float(fms[2]), 4)}
        _log(f"[bench] with a {args.flush_gib} GiB read between steps: stats {fms[0]:.3f} ms, "
             f"select {fms[1]:.3f} ms, attention {fms[2]:.3f} ms")

    # The fused entry point over the same steps (same results, one pass).
    fused_ms = None
    if args.fused_steps > 0:
        fcounts, findices = rbs.allocate_lists(shape, dev)
        Of = torch.empty_like(Q)

        def fstep(ev=None):
            if ev is not None:
                ev[0].record(stream)
            rbs.rbs_block_stats(shape, K, stats, stream=stream)
            if ev is not None:
                ev[1].record(stream)
            rbs.rbs_select_attend(shape, Q, K, V, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local,
                                  w.n_recent, 0.0, fcounts, findices, Of, stream=stream)
            if ev is not None:
                ev[2].record(stream)

        for _ in range(min(args.warmup, 2)):
            fstep()
        fev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.fused_steps)]
        for k in range(args.fused_steps):
            fstep(fev[k])
        torch.cuda.synchronize()
        f = np.zeros(2)
        for ev in fev:
            f += [ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])]
        f /= args.fused_steps
        fused_ms = (float(f[0]), float(f[1]))
        _log(f"[bench] fused path: stats {f[0]:.3f} ms, select+attention {f[1]:.3f} ms "
             f"(total {f.sum():.3f} ms/step)")
        del Of, fcounts, findices

    counts_np = counts.cpu().numpy()
    indices_np = indices.cpu().numpy()
    counts_sum = int(counts_np.sum())
    alg = algorithmic(w, counts_sum)
    density = counts_sum / alg["pairs"]
    causal_flops = exact_causal_flops(w, counts_np)
    sclk_summary = sclk.summary()
    copy_gbps = copy_ceiling_gbps(torch, dev)
    _log(f"[bench] shader clock during the timed steps: {sclk_summary}; 1 GiB copy {copy_gbps:.0f} GB/s")

    # Own dense path: same attention kernel over every causal block.
    dense_ms = None
    if args.dense_reps > 0:
        dense_ms = _time_dense(rbs, torch, np, shape, Q, K, V, stream, args.dense_reps)
        _log(f"[bench] dense attention {dense_ms:.3f} ms")

    # Context for the density: the same layer selected at tighter thresholds.
    # The attention's time follows the executed block pairs; the headline
    # line keeps the workload's own thresholds.
    tau_sweep = None
    if args.tau_sweep:
        tau_sweep = []
        tcounts, tindices = rbs.allocate_lists(shape, dev)
        for tb, tr in TAU_SWEEP:
            rbs.rbs_select(shape, Q, stats, tb, tr, w.n_sink, w.n_local, w.n_recent, tcounts, tindices,
                           stream=stream)
            ts = []
            for _ in range(3):
                a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a_ev.record(stream)
                rbs.rbs_sparse_prefill(shape, Q, K, V, tcounts, tindices, 0.0, O, stream=stream)
                b_ev.record(stream)
                torch.cuda.synchronize()
                ts.append(a_ev.elapsed_time(b_ev))
            t_ms = float(np.median(ts))
            n_exec = int(tcounts.sum().item())
            t_flops = algorithmic(w, n_exec)["attn_flops"]
            tau_sweep.append({"tau_base": tb, "tau_rescue": tr, "density": round(n_exec / alg["pairs"], 6),
                              "attn_ms": round(t_ms, 4),
                              "attn_mfma_frac": round(t_flops / (t_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                              "attn_speedup_vs_dense": round(dense_ms / t_ms, 3) if dense_ms else None})
            _log(f"[bench] tau ({tb}, {tr}): {tau_sweep[-1]}")
        del tcounts, tindices

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    attn_tflops = alg["attn_flops"] / (stage_ms[2] * 1e-3) / 1e12
    dense_tflops = alg["dense_flops"] / (dense_ms * 1e-3) / 1e12 if dense_ms else None
    stats_gbps = alg["stats_bytes"] / (stage_ms[0] * 1e-3) / 1e9
    select_gbps = alg["select_bytes"] / (stage_ms[1] * 1e-3) / 1e9
    select_tflops = alg["select_flops"] / (stage_ms[1] * 1e-3) / 1e12

    traffic = _profiled_traffic("attn_queue_kernel", w.name)

    result = {
        "metric": METRIC,
        "value": round(ms_per_step, 4),
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "seq_len": w.seq_len, "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "block_size": w.block_size, "tau_base": w.tau_base,
                   "tau_rescue": w.tau_rescue, "n_sink": w.n_sink, "n_local": w.n_local,
                   "n_recent": w.n_recent, "seed": w.seed},
        "speedup_vs_dense": round(dense_ms / ms_per_step, 3) if dense_ms else None,
        "attn_speedup_vs_dense": round(dense_ms / stage_ms[2], 3) if dense_ms else None,
        "mfma_util_pct": round(100.0 * attn_tflops / PEAK_BF16_TFLOPS, 2),
        "density": round(density, 6),
        "dense_attn_ms": round(dense_ms, 3) if dense_ms else None,
        "dense_mfma_util_pct": round(100.0 * dense_tflops / PEAK_BF16_TFLOPS, 2) if dense_ms else None,
        "wall_ms_per_step": round(wall_ms, 4),
        "stages": {
            "stats": {"ms": round(float(stage_ms[0]), 4), "median_ms": round(float(stage_med[0]), 4),
                      "alg_bytes": alg["stats_bytes"],
                      "GBps": round(stats_gbps, 1), "hbm_frac": round(stats_gbps / PEAK_HBM_GBPS, 4),
                      "hbm_frac_median": round(alg["stats_bytes"] / (stage_med[0] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)},
            "select": {"ms": round(float(stage_ms[1]), 4), "median_ms": round(float(stage_med[1]), 4),
                       "alg_bytes": alg["select_bytes"],
                       "GBps": round(select_gbps, 1), "hbm_frac": round(select_gbps / PEAK_HBM_GBPS, 4),
                       "alg_flops": alg["select_flops"], "TFLOPs": round(select_tflops, 1),
                       "mfma_frac": round(select_tflops / PEAK_BF16_TFLOPS, 4)},
            "attn": {"ms": round(float(stage_ms[2]), 4), "median_ms": round(float(stage_med[2]), 4),
                     "alg_flops": alg["attn_flops"],
                     "TFLOPs": round(attn_tflops, 1), "executed_pairs": counts_sum,
                     "causal_flops": causal_flops,
                     "exps": counts_sum * w.block_size * w.block_size},
        },
        "flushed": flushed,
        "fused": ({"ms_per_step": round(sum(fused_ms), 4), "stats_ms": round(fused_ms[0], 4),
                   "select_attend_ms": round(fused_ms[1], 4), "steps": args.fused_steps}
                  if fused_ms else None),
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic},
        # Context for the roofline: the shader clock measured while the steps
        # ran (the vendor peak assumes 2.4 GHz) and a plain copy's bandwidth.
        "sclk_mhz": sclk_summary,
        "mfma_frac_at_sclk": (round(attn_tflops / (PEAK_BF16_TFLOPS * sclk_summary["median"] / PEAK_SCLK_MHZ), 4)
                              if sclk_summary else None),
        "copy_GBps": round(copy_gbps, 1),
        "tau_sweep": tau_sweep,
    }

    rates = unit_rates(brief=True)
    if rates is not None:
        result["unit_rates"] = rates

    if not args.no_extra_configs:
        del Q, K, V, O, stats, counts, indices
        torch.cuda.empty_cache()
        result["other_configs"] = {}
        for name in EXTRA_CONFIGS:
            result["other_configs"][name] = _config_line(rbs, torch, np, workload(name), dev)
            _log(f"[bench] {name}: {result['other_configs'][name]}")

    if not args.no_cpu_baseline:
        _log(f"[bench] timing the CPU oracle on sampled rows")
        cb = cpu_baseline(w, inp, counts_np, indices_np, args.cpu_select_rows, args.cpu_attn_rows)
        _log(f"[bench] CPU oracle measured {cb.pop('measured_s'):.1f}s")
        result["cpu_baseline"] = {k: (round(v, 3) if isinstance(v, float) else v) for k, v in cb.items()}
    print(json.dumps(result), flush=True)


# Threshold pairs (tau_base, tau_rescue) of the density context: the
# workload's own, the paper's default pair, then tighter ones (relative
# thresholds closer to 1 keep fewer blocks).
TAU_SWEEP = ((0.9, 0.95), (0.22, 0.18), (0.95, 0.975), (0.97, 0.985), (0.99, 0.995))


# The other workloads of the benchmark's configurations, one compact line
# each: the 128K layer at 64- and 256-token blocks (the block-size
# trade-off), the 32K layer and the 64-head 64K layer.
EXTRA_CONFIGS = ("qwen3-30b-a3b-128k-b64", "qwen3-30b-a3b-128k-b256", "qwen3-30b-a3b-32k", "qwen3-32b-64k")


def _config_line(rbs, torch, np, w, dev, steps: int = 3) -> dict:
    """Stage times (HIP events, mean of `steps` after one warm-up step), the
    attention's executed bf16 rate and the own-dense attention time of one
    workload."""
    from synth import make_inputs
    inp = make_inputs(w)

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    Q, K, V = up(inp["q"]), up(inp["k"]), up(inp["v"])
    del inp
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    stats = rbs.BlockStats.allocate(shape, dev)
    counts, indices = rbs.allocate_lists(shape, dev)
    O = torch.empty_like(Q)
    stream = torch.cuda.current_stream()
    ms = np.zeros(3)
    for k in range(steps + 1):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        rbs.rbs_block_stats(shape, K, stats, stream=stream)
        ev[1].record(stream)
        rbs.rbs_select(shape, Q, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent, counts,
                       indices, stream=stream)
        ev[2].record(stream)
        rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, O, stream=stream)
        ev[3].record(stream)
        torch.cuda.synchronize()
        if k > 0:
            ms += [ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]), ev[2].elapsed_time(ev[3])]
    ms /= steps
    counts_sum = int(counts.sum().item())
    alg = algorithmic(w, counts_sum)
    dense_ms = _time_dense(rbs, torch, np, shape, Q, K, V, stream, 1)
    del Q, K, V, O, stats, counts, indices
    torch.cuda.empty_cache()
    attn_tflops = alg["attn_flops"] / (ms[2] * 1e-3) / 1e12
    return {"ms_per_layer": round(float(ms.sum()), 4), "stats_ms": round(float(ms[0]), 4),
            "select_ms": round(float(ms[1]), 4), "attn_ms": round(float(ms[2]), 4),
            "density": round(counts_sum / alg["pairs"], 6),
            "attn_mfma_frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "stats_hbm_frac": round(alg["stats_bytes"] / (ms[0] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "select_hbm_frac": round(alg["select_bytes"] / (ms[1] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "dense_attn_ms": round(dense_ms, 3), "speedup_vs_dense": round(dense_ms / float(ms.sum()), 3)}


UNIT_RATES_BIN = os.path.join(ROOT, "paper_2609_20971_amd", "rbs_unit_rates")


def unit_rates(brief: bool = False):
    """Run the unit-rate probe (a separate program, built with the library)
    and return its cases; brief: cycles per wave64 instruction of the
    exponential, the FMA and the 32x32x16 bf16 matrix op alone, and the
    matrix op's cycles with the attention's softmax mix beside it."""
    import subprocess
    if not os.path.exists(UNIT_RATES_BIN):
        if brief:
            return None
        raise SystemExit(f"{UNIT_RATES_BIN} is missing: build with `python -m paper_2609_20971_amd.build`")
    out = subprocess.run([UNIT_RATES_BIN], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    if out.returncode != 0:
        if brief:
            return None
        raise SystemExit(f"unit-rate probe failed: {out.stderr}")
    data = json.loads(out.stdout)
    if not brief:
        return data

    def cyc(other, n, w, same=True, mf=0, chains=4):
        for c in data["cases"]:
            if (c["other"] == other and c["n_other"] == n and c["waves_per_simd"] == w and c["mfma"] == mf
                    and c["acc"] == "vgpr" and (c["placement"] == "same_wave") == same
                    and c.get("acc_chains", 4) == chains):
                return c
        return None

    ex, fm, mf = cyc("v_exp_f32", 8, 2), cyc("v_fma_f32", 8, 2), cyc("none", 0, 2, mf=8)
    mix = cyc("softmax_mix", 28, 2, mf=8)
    chain = cyc("none", 0, 1, mf=8, chains=1)  # one wave per SIMD, 8 ops into one accumulator
    # Two waves per SIMD, each issuing 8 of the op (or 8 matrix ops) per loop
    # iteration: one SIMD issues 16 per iteration of either wave.
    per = lambda c: round(c["cycles_per_iter_mfma_wave"] / 16, 2) if c else None
    loop = {c["schedule"]: c["mfma_busy"] for c in data.get("attention_block_loop", [])}
    # LDS read rate of a compute unit: its 4 SIMDs x 2 waves each read 16
    # ops of `size` bytes per iteration (a lower bound: each iteration also
    # waits for its reads).
    lds = lambda c, size: round(4 * 2 * 16 * size / c["cycles_per_iter_mfma_wave"], 1) if c else None
    return {"exp_cycles": per(ex), "fma_cycles": per(fm), "mfma_32x32x16_bf16_cycles": per(mf),
            "mfma_cycles_with_softmax_mix": per(mix),
            "mfma_cycles_dependent_chain": (round(chain["cycles_per_iter_mfma_wave"] / 8, 2) if chain else None),
            "lds_read_bytes_per_clk_per_cu": {"ds_read_b128": lds(cyc("ds_read_b128", 16, 2), 1024),
                                              "ds_read_b64_tr_b16": lds(cyc("ds_read_b64_tr_b16", 16, 2), 512)},
            "block_loop_mfma_busy": loop or None,
            "note": "shader-clock cycles one SIMD spends per wave64 instruction, two waves per SIMD; "
                    "the mix is 28 exp/fma/max/convert ops beside each 8 matrix ops in the same wave; "
                    "dependent_chain: one wave per SIMD, each matrix op accumulating into the previous one's "
                    "result; "
                    "lds: bytes per shader clock one compute unit's LDS returned to 8 waves reading "
                    "conflict-free words; block_loop: busy fraction of the matrix unit over the 64 QK^T and "
                    "PV ops per block of the attention's block loop on LDS-resident tiles (one workgroup "
                    "per CU; denominator on the matrix core, as the kernel): free-running, as a barrier "
                    "ping-pong, with one wave per SIMD, with 64-key softmax steps at two and three waves "
                    "per SIMD, and free-running with the denominator summed by v_dot2"}


def _time_dense(rbs, torch, np, shape, Q, K, V, stream, reps: int) -> float:
    """Median time of the attention kernel over every causal block (the
    build's own dense path), HIP events on the launch stream."""
    dcounts, dindices = rbs.allocate_lists(shape, Q.device)
    rbs.rbs_dense_indices(shape, dcounts, dindices, stream=stream)
    Od = torch.empty_like(Q)
    rbs.rbs_sparse_prefill(shape, Q, K, V, dcounts, dindices, 0.0, Od, stream=stream)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        rbs.rbs_sparse_prefill(shape, Q, K, V, dcounts, dindices, 0.0, Od, stream=stream)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    del Od, dcounts, dindices
    return float(np.median(times))


# Selector study: each selector's parameter is calibrated by bisection to
# these actual densities (the paper aligns its selector comparison by measured
# density), and the named settings are reported as they are: the benchmark and
# the paper's default threshold pairs, and the paper's comparison settings of
# the single-branch selectors (0.194, 0.022, budget 0.0405).
STUDY_TARGETS = (0.05, 0.10, 0.20, 0.40)
STUDY_NAMED = [("rbs", (0.9, 0.95)), ("rbs", (0.22, 0.18)), ("centroid", 0.194), ("full_l2", 0.022),
               ("box", 0.0405)]


def selector_study(args):
    """Synthetic analogue of the paper's selected-block-ratio vs attention-mass
    comparison and of its selector comparison: per selector and density, the
    recall of planted needles (the needle's key block is in the list of its
    target query head and query block) and the mean fraction of the dense
    causal softmax mass of sampled query blocks that falls in their selected
    key blocks."""
    import numpy as np
    import torch

    import paper_2609_20971_amd as rbs
    from synth import workload, make_inputs

    w = workload(args.workload or "qwen3-30b-a3b-32k")
    if args.study_needle_norm is not None:
        w = w.with_(needle_norm=args.study_needle_norm)
    inp = make_inputs(w)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(0)

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    Q, K = up(inp["q"]), up(inp["k"])
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    stats = rbs.rbs_block_stats(shape, K)
    box = rbs.rbs_block_box(shape, K)
    B, M, N, G = w.block_size, w.n_blocks, w.seq_len, w.group
    pairs = w.n_q_heads * M * (M + 1) / 2
    rng = np.random.default_rng(1)
    rows = sorted({(int(rng.integers(w.n_q_heads)), int(rng.integers(4, M))) for _ in range(args.study_rows)})
    _log(f"[study] {w.name}: needle norm {w.needle_norm}, {len(rows)} sampled rows, {len(inp['needles'])} needles")

    # Dense causal softmax mass per key block, averaged over each sampled row's queries.
    scale = 1.0 / float(np.sqrt(w.head_dim))
    mass = {}
    for (h, i) in rows:
        q0, q1 = i * B, min((i + 1) * B, N)
        s = (Q[h, q0:q1].float() @ K[h // G, :q1].float().t().contiguous()) * scale
        pos = torch.arange(q1, device=dev)
        p = torch.softmax(s.masked_fill(pos[None, :] > pos[q0:q1, None], float("-inf")), dim=1)
        blocks = torch.zeros((q1 - q0, i + 1), device=dev)
        blocks.index_add_(1, pos // B, p)
        mass[(h, i)] = blocks.mean(dim=0).cpu().numpy()

    counts, idx = rbs.allocate_lists(shape, dev)

    def run(name, param):
        if name == "rbs":
            tb, tr = param if isinstance(param, tuple) else (param, param)
            rbs.rbs_select(shape, Q, stats, tb, tr, w.n_sink, w.n_local, w.n_recent, counts, idx)
        else:
            rbs.rbs_select_variant(shape, Q, stats, name, param, w.n_sink, w.n_local, w.n_recent, box=box,
                                   counts=counts, indices=idx)
        return float(counts.sum().item()) / pairs

    def calibrate(name, target):
        # Density falls as a relative threshold rises and grows with a budget:
        # bisect the threshold in log(1 - tau) (it matters near 1) or log(tau)
        # below 0.5, and the budget in log space.
        if name == "box":
            lo, hi = 1e-4, 1.0
            for _ in range(30):
                mid = (lo * hi) ** 0.5
                if run(name, mid) < target: lo = mid
                else: hi = mid
            return hi
        lo, hi = -87.0, 30.0  # tau = sigmoid(x) down to ~1e-38 (float32); x -> +inf keeps the argmax
        for _ in range(40):
            mid = 0.5 * (lo + hi)
            if run(name, float(1.0 / (1.0 + np.exp(-mid)))) > target: lo = mid
            else: hi = mid
        return float(1.0 / (1.0 + np.exp(-lo)))

    def evaluate(name, param, target):
        density = run(name, param)
        cnt = counts.cpu().numpy()
        ind = idx.cpu().numpy()

        def row_list(h, i):
            off = i * (i + 1) // 2
            return ind[h, off:off + cnt[h, i]]

        hits = [int(p // B) in set(row_list(h, j // B).tolist()) for (g, p, h, j) in inp["needles"]]
        recall = float(np.mean(hits)) if hits else None
        cover = float(np.mean([mass[(h, i)][row_list(h, i)].sum() for (h, i) in rows]))
        pt = {"selector": name, "param": list(param) if isinstance(param, tuple) else float(param),
              "target": target, "density": round(density, 5),
              "target_reached": None if target is None else bool(abs(density - target) <= 0.05 * target),
              "needle_recall": None if recall is None else round(recall, 4), "mass_coverage": round(cover, 5)}
        _log(f"[study] {name:8s} {'' if target is None else f'target {target:.2f}':12s} param "
             f"{str(pt['param']):26s} density {density:7.4f}  needle recall {pt['needle_recall']}  "
             f"mass coverage {cover:.4f}")
        return pt

    points = []
    for name in ("rbs", "centroid", "full_l2", "box"):
        for target in STUDY_TARGETS:
            points.append(evaluate(name, calibrate(name, target), target))
    for name, param in STUDY_NAMED:
        points.append(evaluate(name, param, None))
    print(json.dumps({"study": "selector comparison", "workload": w.name, "needle_norm": w.needle_norm,
                      "rows": len(rows), "needles": len(inp["needles"]), "points": points}), flush=True)


def _upload(torch, np, bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)


def _events(torch, n):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def batch_bench(args):
    """A batch of independent sequences (the paper's batched prompt throughput:
    separate causal sequences, normalized to dense at the same batch): the
    varlen calls (one launch per stage for the whole batch) against the same
    sequences run one single-sequence call at a time, and the dense path of
    the varlen attention.  One JSON line."""
    import numpy as np
    import torch

    import paper_2609_20971_amd as rbs
    from synth import workload, batch_workloads, make_batch_inputs

    w = workload(args.workload or "qwen3-30b-a3b-128k")
    lens = ([int(x) for x in args.batch_lens.split(",")] if args.batch_lens else [w.seq_len] * args.batch)
    per_2k = w.needles_per_kv_head * 2048 / w.seq_len
    t0 = time.perf_counter()
    inp = make_batch_inputs(batch_workloads(w, lens, needles_per_2k=per_2k))
    _log(f"[batch] {w.name} x {len(lens)}: lengths {lens}; inputs in {time.perf_counter() - t0:.1f}s")
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(0)
    Q, K, V = (_upload(torch, np, inp[x], dev) for x in ("q", "k", "v"))
    batch = rbs.Batch(lens)
    shape = rbs.varlen_shape(batch, w.n_q_heads, w.n_kv_heads, w.block_size)
    stats = rbs.allocate_stats_varlen(shape, batch, dev)
    counts, indices = rbs.allocate_lists_varlen(shape, batch, dev)
    O = torch.empty_like(Q)
    stream = torch.cuda.current_stream()
    tb, tr, sink, local, recent = w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent

    def varlen_step():
        rbs.rbs_block_stats_varlen(shape, batch, K, stats, stream=stream)
        rbs.rbs_select_varlen(shape, batch, Q, stats, tb, tr, sink, local, recent, counts, indices, stream=stream)
        rbs.rbs_sparse_prefill_varlen(shape, batch, Q, K, V, counts, indices, 0.0, O, stream=stream)

    # The same sequences one at a time through the single-sequence calls, on
    # views of the packed tensors copied out once (outside the timed region).
    off = batch.token_offsets()
    singles = []
    for s_, n in enumerate(lens):
        sh = rbs.make_shape(n, w.n_q_heads, w.n_kv_heads, w.block_size)
        q, k, v = (X[:, off[s_]:off[s_ + 1]].contiguous() for X in (Q, K, V))
        singles.append((sh, q, k, v, rbs.BlockStats.allocate(sh, dev), *rbs.allocate_lists(sh, dev),
                        torch.empty_like(q)))

    def single_step():
        for (sh, q, k, v, st, c, ix, o) in singles:
            rbs.rbs_block_stats(sh, k, st, stream=stream)
            rbs.rbs_select(sh, q, st, tb, tr, sink, local, recent, c, ix, stream=stream)
            rbs.rbs_sparse_prefill(sh, q, k, v, c, ix, 0.0, o, stream=stream)

    dcounts, dindices = rbs.allocate_lists_varlen(shape, batch, dev)
    rbs.rbs_dense_indices_varlen(shape, batch, dcounts, dindices, stream=stream)

    def dense_step():
        rbs.rbs_sparse_prefill_varlen(shape, batch, Q, K, V, dcounts, dindices, 0.0, O, stream=stream)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a, b = _events(torch, 2)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    reps = max(1, args.steps)
    t_var = timed(varlen_step, reps)
    _log(f"[batch] varlen: {t_var:.3f} ms per batch")
    t_single = timed(single_step, reps)
    _log(f"[batch] one sequence at a time: {t_single:.3f} ms per batch")
    t_dense = timed(dense_step, max(1, args.dense_reps))
    _log(f"[batch] dense attention (varlen): {t_dense:.3f} ms per batch")
    csum = int(counts.sum().item())
    pairs = w.n_q_heads * sum(m * (m + 1) // 2 for m in batch.block_counts(w.block_size))
    tokens = batch.n_tokens
    print(json.dumps({
        "mode": "batch", "workload": w.name, "seq_tokens": lens, "n_seqs": len(lens), "dtype": "bf16",
        "data": "synthetic", "steps": reps,
        "varlen_ms_per_batch": round(t_var, 4), "single_calls_ms_per_batch": round(t_single, 4),
        "dense_attn_ms_per_batch": round(t_dense, 4),
        "prompt_tokens_per_s": round(tokens / (t_var * 1e-3), 1),
        "throughput_vs_dense": round(t_dense / t_var, 3),
        "varlen_vs_single_calls": round(t_single / t_var, 3),
        "density": round(csum / pairs, 6),
    }), flush=True)


PEAK_FP8_TFLOPS = 5000.0     # MI355X dense FP8 MFMA, vendor figure (no sparsity)


def fp8_bench(args):
    """Attention on FP8 (E4M3) copies of Q, K, V (rbs_sparse_prefill_fp8) over
    the selector's lists of the 128K layer, timed against the bf16 attention on
    the same lists and against the FP8 dense path; the packing (amax + E4M3
    conversion) is timed on its own, since an FP8 model's K/V cache is already
    FP8.  One JSON line."""
    import numpy as np
    import torch

    import paper_2609_20971_amd as rbs
    from synth import workload, make_inputs

    w = workload(args.workload or "qwen3-30b-a3b-128k")
    inp = make_inputs(w)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(0)
    Q, K, V = (_upload(torch, np, inp[x], dev) for x in ("q", "k", "v"))
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    stream = torch.cuda.current_stream()
    stats = rbs.rbs_block_stats(shape, K, stream=stream)
    counts, indices = rbs.rbs_select(shape, Q, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent,
                                     stream=stream)
    f8 = rbs.allocate_fp8(shape, dev)
    O = torch.empty_like(Q)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a, b = _events(torch, 2)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    reps = max(1, args.steps)
    t_pack = timed(lambda: rbs.rbs_fp8_prepare(shape, Q, K, V, f8, stream=stream), reps)
    t_f8 = timed(lambda: rbs.rbs_sparse_prefill_fp8(shape, f8, counts, indices, 0.0, O, stream=stream), reps)
    t_bf = timed(lambda: rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, O, stream=stream), reps)
    dc, di = rbs.rbs_dense_indices(shape, device=dev)
    t_f8d = timed(lambda: rbs.rbs_sparse_prefill_fp8(shape, f8, dc, di, 0.0, O, stream=stream),
                  max(1, args.dense_reps))
    csum = int(counts.sum().item())
    alg = algorithmic(w, csum)
    tf_f8 = alg["attn_flops"] / (t_f8 * 1e-3) / 1e12
    tf_f8d = alg["dense_flops"] / (t_f8d * 1e-3) / 1e12
    _log(f"[fp8] pack {t_pack:.3f} ms; attention fp8 {t_f8:.3f} ms ({tf_f8:.0f} TFLOP/s) vs bf16 {t_bf:.3f} ms; "
         f"fp8 dense {t_f8d:.3f} ms ({tf_f8d:.0f} TFLOP/s)")
    print(json.dumps({
        "mode": "fp8", "workload": w.name, "dtype": "fp8 e4m3 (Q, K, V, P); fp32 accumulate", "data": "synthetic",
        "steps": reps, "density": round(csum / alg["pairs"], 6),
        "pack_ms": round(t_pack, 4), "attn_fp8_ms": round(t_f8, 4), "attn_bf16_ms": round(t_bf, 4),
        "attn_fp8_vs_bf16": round(t_bf / t_f8, 3),
        "attn_fp8_tflops": round(tf_f8, 1), "attn_fp8_mfma_frac": round(tf_f8 / PEAK_FP8_TFLOPS, 4),
        "dense_fp8_ms": round(t_f8d, 3), "dense_fp8_tflops": round(tf_f8d, 1),
        "dense_fp8_mfma_frac": round(tf_f8d / PEAK_FP8_TFLOPS, 4),
    }), flush=True)


def layer_sweep(args):
    """The 48-layer prefill sweep of the 128K layer (per-layer key noise and
    needle counts from the seeded layer schedule, so density varies by layer):
    per-layer density, sparse path and dense attention times, totals; then the
    whole sweep again with layer l+1's statistics and selection issued on a
    second stream while layer l's attention runs.  One JSON line."""
    import numpy as np
    import torch

    import paper_2609_20971_amd as rbs
    from synth import layer_schedule, make_inputs

    layers = layer_schedule(args.layer_sweep)
    w0 = layers[0]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(0)
    shape = rbs.make_shape(w0.seq_len, w0.n_q_heads, w0.n_kv_heads, w0.block_size)
    t0 = time.perf_counter()
    data = []
    for lw in layers:  # every layer's Q, K, V resident in HBM (about 1.3 GB per layer)
        inp = make_inputs(lw)
        data.append(tuple(_upload(torch, np, inp[x], dev) for x in ("q", "k", "v")))
        del inp
        _log(f"[sweep] {lw.name}: key sigma {lw.key_noise[0][1]:.3f}, {lw.needles_per_kv_head} needles / KV head "
             f"({time.perf_counter() - t0:.0f}s)")
    main_s = torch.cuda.current_stream()
    side_s = torch.cuda.Stream()
    sets = [(rbs.BlockStats.allocate(shape, dev), *rbs.allocate_lists(shape, dev)) for _ in range(2)]
    O = torch.empty_like(data[0][0])
    tb, tr, sink, local, recent = w0.tau_base, w0.tau_rescue, w0.n_sink, w0.n_local, w0.n_recent

    def select_layer(l, st, c, ix, stream):
        Q, K, _ = data[l]
        rbs.rbs_block_stats(shape, K, st, stream=stream)
        rbs.rbs_select(shape, Q, st, tb, tr, sink, local, recent, c, ix, stream=stream)

    # Serial pass, stage events per layer.
    st, c, ix = sets[0]
    select_layer(0, st, c, ix, main_s)
    rbs.rbs_sparse_prefill(shape, *data[0], c, ix, 0.0, O, stream=main_s)
    torch.cuda.synchronize()
    ev = [_events(torch, 3) for _ in layers]
    dens = []
    t_start = time.perf_counter()
    for l in range(len(layers)):
        ev[l][0].record(main_s)
        select_layer(l, st, c, ix, main_s)
        ev[l][1].record(main_s)
        rbs.rbs_sparse_prefill(shape, *data[l], c, ix, 0.0, O, stream=main_s)
        ev[l][2].record(main_s)
        dens.append(c.sum())
    torch.cuda.synchronize()
    serial_wall = (time.perf_counter() - t_start) * 1e3
    sel_ms = [e[0].elapsed_time(e[1]) for e in ev]
    att_ms = [e[1].elapsed_time(e[2]) for e in ev]
    pairs = w0.n_q_heads * w0.n_blocks * (w0.n_blocks + 1) // 2
    density = [float(d.item()) / pairs for d in dens]
    _log(f"[sweep] serial: {sum(sel_ms) + sum(att_ms):.1f} ms ({serial_wall:.1f} ms wall)")

    # Dense attention per layer.
    dc, di = rbs.rbs_dense_indices(shape, device=dev)
    dense_ms = []
    for l in range(len(layers)):
        a, b = _events(torch, 2)
        a.record(main_s)
        rbs.rbs_sparse_prefill(shape, *data[l], dc, di, 0.0, O, stream=main_s)
        b.record(main_s)
        b.synchronize()
        dense_ms.append(a.elapsed_time(b))
    _log(f"[sweep] dense attention: {sum(dense_ms):.1f} ms")
    del dc, di

    # Pipelined pass: layer l+1's stats and selection on the side stream while
    # layer l's attention runs on the main stream (double-buffered summaries
    # and lists; events order every hand-off).
    ready = [torch.cuda.Event() for _ in layers]
    done = [torch.cuda.Event() for _ in layers]
    torch.cuda.synchronize()
    a, b = _events(torch, 2)
    a.record(main_s)
    side_s.wait_event(a)
    select_layer(0, *sets[0], side_s)
    ready[0].record(side_s)
    for l in range(len(layers)):
        if l + 1 < len(layers):
            if l >= 1:
                side_s.wait_event(done[l - 1])  # layer l-1's attention has read set (l+1) % 2
            select_layer(l + 1, *sets[(l + 1) % 2], side_s)
            ready[l + 1].record(side_s)
        st, c, ix = sets[l % 2]
        main_s.wait_event(ready[l])
        rbs.rbs_sparse_prefill(shape, *data[l], c, ix, 0.0, O, stream=main_s)
        done[l].record(main_s)
    b.record(main_s)
    torch.cuda.synchronize()
    piped_ms = a.elapsed_time(b)
    _log(f"[sweep] pipelined: {piped_ms:.1f} ms")
    total_sparse = sum(sel_ms) + sum(att_ms)
    print(json.dumps({
        "mode": "layer_sweep", "layers": len(layers), "workload": w0.name.rsplit("-layer", 1)[0],
        "dtype": "bf16", "data": "synthetic",
        "density": [round(x, 5) for x in density],
        "select_ms": [round(x, 3) for x in sel_ms], "attn_ms": [round(x, 3) for x in att_ms],
        "dense_attn_ms": [round(x, 3) for x in dense_ms],
        "total_sparse_ms": round(total_sparse, 2), "total_dense_attn_ms": round(sum(dense_ms), 2),
        "speedup_vs_dense": round(sum(dense_ms) / total_sparse, 3),
        "pipelined_total_ms": round(piped_ms, 2),
        "mean_density": round(float(np.mean(density)), 5),
    }), flush=True)


# Sources each kernel is built from, with the build script (it holds per-source
# compiler flags); their joint hash identifies the kernel in the committed
# rocprofv3 summaries.  The attention calls run the persistent (queue) kernels.
KERNEL_SOURCES = {
    "stats_kernel": ["stats.hip", "rbs_device.hpp", "../build.py"],
    "quantile_kernel": ["stats.hip", "rbs_device.hpp", "../build.py"],
    "select_kernel": ["select.hip", "select_block.hpp", "rbs_device.hpp", "../build.py"],
    "attn_queue_kernel": ["attn.hip", "attend_block.hpp", "rbs_device.hpp", "rbs_launch.hpp", "../build.py"],
    "select_attend_queue_kernel": ["fused.hip", "select_block.hpp", "attend_block.hpp", "rbs_device.hpp",
                                   "rbs_launch.hpp", "../build.py"],
    "attn_fp8_queue_kernel": ["fp8.hip", "attend_block.hpp", "rbs_device.hpp", "rbs_launch.hpp", "../build.py"],
}


def source_sha(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for src in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_20971_amd", "csrc", src), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _profiled_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 summary of this kernel
    on this workload, or None when there is none or the kernel sources changed
    since the counters were taken."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ": " in line and not line.startswith(" "):
                k, v = line.split(": ", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_sha") != source_sha(kernel) or "traffic_bytes_per_launch" not in fields:
        return None
    return int(float(fields["traffic_bytes_per_launch"]))


if __name__ == "__main__":
    main()
