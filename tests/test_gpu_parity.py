"""GPU parity: the HIP path through the C ABI against the float64 oracle on the
same seeded inputs.  Tolerances live in tests/rbs_harness.py."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, Workload, f64_from_bf16_bits, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run(w: Workload, inputs=None, tau=None, forced=None):
    import torch
    import paper_2609_20971_amd as rbs
    if inputs is None:
        inputs = make_inputs(w)
    tb, tr = (w.tau_base, w.tau_rescue) if tau is None else tau
    sink, local, recent = (w.n_sink, w.n_local, w.n_recent) if forced is None else forced
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Qd, Kd, Vd = (H.to_device(inputs[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats(shape, Kd)
    counts, indices = rbs.rbs_select(shape, Qd, st, tb, tr, sink, local, recent)
    lse = torch.empty((w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    O = rbs.rbs_sparse_prefill(shape, Qd, Kd, Vd, counts, indices, 0.0, lse=lse)
    torch.cuda.synchronize()
    return dict(shape=shape, inputs=inputs, Qd=Qd, Kd=Kd, Vd=Vd, stats=st, counts=counts, indices=indices,
                O=O, lse=lse, tau=(tb, tr), forced=(sink, local, recent))


def _oracle_check(w: Workload, inp, counts, indices, O, tau, forced, rows=None, attn_rows=None, label=None):
    """Lists and O of one HIP call against the oracle: masks bit for bit outside
    the near-threshold band, the lists' structure, and O on the GPU's own lists
    within the attention tolerance.  Returns (near-threshold flips, density)."""
    Kf = f64_from_bf16_bits(inp["k"])
    C, R = oracle.block_stats(Kf, w.block_size)
    beta, _ = oracle.rescue_coefficients(R)
    M = w.n_blocks
    rows = rows or [(h, i) for h in range(w.n_q_heads) for i in range(M)]
    Qf = f64_from_bf16_bits(inp["q"])
    tb, tr = tau
    sink, local, recent = forced
    ref = oracle.select(Qf, C, R, beta, w.block_size, tb, tr, sink, local, recent, rows=rows)
    lists = H.gpu_rows(counts, indices, rows)
    H.check_lists(lists, M, sink, local, recent)
    n_rows, compared, near = H.compare_masks(lists, ref)
    dens_gpu = sum(len(v) for v in lists.values()) / compared
    dens_ref = oracle.density([ref[k]["final"] for k in rows])
    arows = attn_rows or rows
    alists = H.gpu_rows(counts, indices, arows)
    Og = H.bf16_tensor_to_f64(O)
    Vf = f64_from_bf16_bits(inp["v"])
    err = H.max_abs_attention_error(Og, Qf, Kf, Vf, w.group, w.block_size, alists, w.seq_len)
    _say(f"[parity] {label or w.name}: rows {n_rows} blocks {compared} near-threshold flips {near}; "
         f"density gpu {dens_gpu:.4f} oracle {dens_ref:.4f}; attention max-abs {err:.3e} ({len(arows)} rows)")
    assert err <= H.ATTN_ATOL
    return near, dens_gpu


def _full_check(w: Workload, tau=None, forced=None, attn_rows=None, select_rows=None, inputs=None):
    _say(f"[parity] workload={w.name} N={w.seq_len} Hq={w.n_q_heads} Hkv={w.n_kv_heads} B={w.block_size} "
         f"tau={tau} forced={forced}")
    r = _run(w, inputs=inputs, tau=tau, forced=forced)
    inp = r["inputs"]
    Kf = f64_from_bf16_bits(inp["k"])
    C, R = oracle.block_stats(Kf, w.block_size)
    beta, rq = oracle.rescue_coefficients(R)
    rep = H.check_stats(r["stats"], C, R, beta, rq)
    _say(f"[parity] {w.name}: stats {rep}")
    near, _ = _oracle_check(w, inp, r["counts"], r["indices"], r["O"], r["tau"], r["forced"], rows=select_rows,
                            attn_rows=attn_rows)
    return r, near


def test_tiny_workload_full():
    _full_check(WORKLOADS["tiny-2k"])


@pytest.mark.parametrize("variant", [
    dict(seq_len=1000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=1),          # ragged tail, GQA 2:1
    dict(seq_len=777, block_size=128, n_q_heads=2, n_kv_heads=2, seed=2),          # no GQA, ragged
    dict(seq_len=1300, block_size=256, n_q_heads=4, n_kv_heads=1, seed=3),         # B = 256, ragged
    dict(seq_len=64, block_size=64, n_q_heads=2, n_kv_heads=1, seed=4),            # single block
    dict(seq_len=5, block_size=128, n_q_heads=1, n_kv_heads=1, seed=5),            # N < B
])
def test_edge_shapes(variant):
    w = WORKLOADS["tiny-2k"].with_(name="edge", needles_per_kv_head=2, **variant)
    _full_check(w)


@pytest.mark.parametrize("variant", [
    dict(seq_len=6000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=11),         # 94 blocks, ragged
    dict(seq_len=9000, block_size=256, n_q_heads=4, n_kv_heads=1, seed=12),        # 36 blocks, two softmax steps per block
    dict(seq_len=8191, block_size=128, n_q_heads=8, n_kv_heads=2, seed=13),        # 64 blocks, one row short
    # 266 blocks at B = 64: late rows list their candidates in three 128-block
    # chunks, the last one partial (block masks spanning chunk ends).
    dict(seq_len=17000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=14),
])
def test_multiblock_rows(variant):
    """Rows spanning many key blocks at every block size: selection on all rows,
    attention on a sample that includes the ragged last row."""
    w = WORKLOADS["tiny-2k"].with_(name="multiblock", needles_per_kv_head=6, **variant)
    M = w.n_blocks
    attn = H.sample_rows(w.n_q_heads, M, 16, seed=variant["seed"], include=[(0, M - 1), (w.n_q_heads - 1, M - 2)])
    _full_check(w, attn_rows=attn)


@pytest.mark.parametrize("tau,forced", [
    ((0.0, 0.0), (1, 2, 0)),     # alpha = 0: every causal block
    ((1.0, 1.0), (0, 1, 0)),     # alpha = 1: argmax blocks only
    ((0.22, 0.18), (1, 2, 0)),   # the paper's default pair
    ((0.9, 0.95), (2, 3, 1)),    # one recent row
    ((0.9, 0.95), (0, 1, 2)),    # two recent rows
])
def test_threshold_and_forced_variants(tau, forced):
    w = WORKLOADS["tiny-2k"].with_(seq_len=1536, seed=7)
    r, _ = _full_check(w, tau=tau, forced=forced)
    if tau == (0.0, 0.0):
        counts = r["counts"].cpu().numpy()
        assert (counts == np.arange(w.n_blocks)[None, :] + 1).all()


def test_degenerate_radii_and_zero_queries():
    """Identical key blocks (r_high == r_low) and all-zero query rows."""
    w = WORKLOADS["tiny-2k"].with_(seq_len=1024, seed=8)
    inp = make_inputs(w)
    blk = inp["k"][:, :w.block_size].copy()
    inp["k"][:] = np.tile(blk, (1, w.seq_len // w.block_size, 1))
    inp["q"][:, 128:320] = 0
    _full_check(w, inputs=inp)


def _scaled(bits, factor):
    from synth import bf16_bits_from_f32, f32_from_bf16_bits
    return bf16_bits_from_f32(f32_from_bf16_bits(bits) * np.float32(factor))


def test_large_norm_queries_take_the_shifted_selector_path():
    """Queries 40x larger: |q| |c'| exceeds the unshifted-sum bound in every
    tile, so every block sum takes the maximum-shifted path."""
    w = WORKLOADS["tiny-2k"].with_(seq_len=1536, seed=31)
    inp = make_inputs(w)
    inp["q"] = _scaled(inp["q"], 40.0)
    _full_check(w, inputs=inp)


def test_mixed_shifted_and_unshifted_tiles():
    """A few key blocks of the second 32-block tile 60x larger: rows past
    block 32 score that tile on the shifted path and the others unshifted."""
    w = WORKLOADS["tiny-2k"].with_(name="mixed", seq_len=6000, block_size=64, n_q_heads=4, n_kv_heads=2,
                                   needles_per_kv_head=4, seed=32)
    inp = make_inputs(w)
    for b in (40, 45):
        inp["k"][:, b * 64:(b + 1) * 64] = _scaled(inp["k"][:, b * 64:(b + 1) * 64], 60.0)
    M = w.n_blocks
    attn = H.sample_rows(w.n_q_heads, M, 12, seed=5, include=[(0, M - 1), (3, 45), (1, 20)])
    _full_check(w, inputs=inp, attn_rows=attn)


def test_unshifted_sums_at_the_bound_b256():
    """B = 256 (a block's sum adds eight waves' partial sums), every query
    aligned with the longest select-ready centroid and scaled so that
    |q| max_b |c'_b| sits just under the unshifted-sum bound (112, log2
    units): the block of that centroid sums 256 terms near 2^108 each, which
    must stay finite; in the attention, later blocks exceed the fixed softmax
    reference (taken from the sink block) by far more than fp32's exponent
    range near 1, which its power-of-two rescales absorb without a restart."""
    from synth import bf16_bits_from_f32, f64_from_bf16_bits
    w = WORKLOADS["tiny-2k"].with_(name="bound", seq_len=2048, block_size=256, n_q_heads=2, n_kv_heads=1,
                                   needles_per_kv_head=2, seed=33)
    inp = make_inputs(w)
    K = f64_from_bf16_bits(inp["k"])[0]
    cent = K.reshape(w.n_blocks, w.block_size, -1).mean(axis=1) * (np.log2(np.e) / np.sqrt(w.head_dim))
    norms = np.linalg.norm(cent, axis=1)
    b_star = int(np.argmax(norms))
    q = cent[b_star] / norms[b_star] * (108.0 / norms[b_star])
    inp["q"] = np.ascontiguousarray(np.broadcast_to(bf16_bits_from_f32(q.astype(np.float32)), inp["q"].shape))
    _say(f"[parity] bound case: block {b_star}, |q| max|c'| = {np.linalg.norm(q) * norms[b_star]:.2f}")
    M = w.n_blocks
    _full_check(w, inputs=inp, attn_rows=H.sample_rows(w.n_q_heads, M, 4, seed=3, include=[(0, M - 1), (1, b_star)]))


def test_dense_path_matches_dense_oracle():
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(seq_len=640, seed=9)
    _say(f"[parity] dense path N={w.seq_len}")
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Qd, Kd, Vd = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    counts, indices = rbs.rbs_dense_indices(shape)
    O = rbs.rbs_sparse_prefill(shape, Qd, Kd, Vd, counts, indices)
    torch.cuda.synchronize()
    Og = H.bf16_tensor_to_f64(O)
    Qf, Kf, Vf = (f64_from_bf16_bits(inp[x]) for x in ("q", "k", "v"))
    for h in range(w.n_q_heads):
        ref = oracle.dense_causal_attention(Qf[h], Kf[h // w.group], Vf[h // w.group])
        assert np.abs(Og[h] - ref).max() <= H.ATTN_ATOL


def test_lse_and_determinism():
    import torch
    w = WORKLOADS["tiny-2k"].with_(seq_len=1152, seed=10)
    r1 = _run(w)
    r2 = _run(w, inputs=r1["inputs"])
    for key in ("counts", "O", "lse"):
        assert torch.equal(r1[key], r2[key]), key
    assert torch.equal(r1["stats"].centroids, r2["stats"].centroids)
    cnt = r1["counts"].cpu().numpy()
    idx = r1["indices"].cpu().numpy()
    for h in range(w.n_q_heads):
        for i in range(w.n_blocks):
            base = i * (i + 1) // 2
            assert (idx[h, base:base + cnt[h, i]] == r2["indices"].cpu().numpy()[h, base:base + cnt[h, i]]).all()
    # LSE of a sampled row against the oracle definition on the GPU's list.
    Qf, Kf = (f64_from_bf16_bits(r1["inputs"][x]) for x in ("q", "k"))
    h, i = 1, w.n_blocks - 1
    base = i * (i + 1) // 2
    ids = idx[h, base:base + cnt[h, i]]
    keys = np.concatenate([np.arange(b * w.block_size, (b + 1) * w.block_size) for b in ids])
    lse = r1["lse"].cpu().numpy()
    for t in range(i * w.block_size, (i + 1) * w.block_size, 17):
        kk = keys[keys <= t]
        x = Kf[0, kk] @ Qf[h, t] / np.sqrt(128)
        ref = x.max() + np.log(np.exp(x - x.max()).sum())
        assert abs(lse[h, t] - ref) <= 1e-3


@pytest.mark.slow
def test_qwen3_30b_32k_select_full_attention_sampled():
    w = WORKLOADS["qwen3-30b-a3b-32k"]
    rows_attn = H.sample_rows(w.n_q_heads, w.n_blocks, 12, seed=1)
    _full_check(w, attn_rows=rows_attn)


@pytest.mark.slow
def test_qwen3_30b_128k_sampled():
    """The headline shape, in the launch configuration the benchmark times;
    selection and attention checked on sampled rows."""
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["qwen3-30b-a3b-128k"]
    rows = H.sample_rows(w.n_q_heads, w.n_blocks, 96, seed=2, include=[(5, 1023), (31, 700), (0, 3)])
    attn = H.sample_rows(w.n_q_heads, w.n_blocks, 12, seed=7, include=[(5, 1023), (31, 700), (0, 3)])
    r, _ = _full_check(w, select_rows=rows, attn_rows=attn)
    # Every row's list, not only the sampled ones: ascending, unique, causal,
    # holding the forced blocks.
    every = [(h, i) for h in range(w.n_q_heads) for i in range(w.n_blocks)]
    H.check_lists(H.gpu_rows(r["counts"], r["indices"], every), w.n_blocks, w.n_sink, w.n_local, w.n_recent)
    _say(f"[parity] {w.name}: all {len(every)} lists well formed")
    # The benchmark's (persistent) launch against one workgroup per (head,
    # query block) on the same lists: every output bit identical.
    lse = torch.empty_like(r["lse"])
    O = rbs.rbs_sparse_prefill(r["shape"], r["Qd"], r["Kd"], r["Vd"], r["counts"], r["indices"], 0.0, lse=lse,
                               workspace=None)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), r["O"].view(torch.int16))
    assert torch.equal(lse, r["lse"])
    _say(f"[parity] {w.name}: persistent and per-item launches bit-identical")


@pytest.mark.slow
def test_qwen3_30b_128k_low_density_sampled():
    """The headline layer at tighter thresholds (3% density, near the paper's
    operating point): sampled rows against the oracle, every list well formed."""
    w = WORKLOADS["qwen3-30b-a3b-128k"]
    tau = (0.95, 0.975)
    rows = H.sample_rows(w.n_q_heads, w.n_blocks, 48, seed=5, include=[(7, 1023), (20, 512)])
    attn = H.sample_rows(w.n_q_heads, w.n_blocks, 8, seed=6, include=[(7, 1023)])
    r, _ = _full_check(w, tau=tau, select_rows=rows, attn_rows=attn)
    every = [(h, i) for h in range(w.n_q_heads) for i in range(w.n_blocks)]
    lists = H.gpu_rows(r["counts"], r["indices"], every)
    H.check_lists(lists, w.n_blocks, w.n_sink, w.n_local, w.n_recent)
    density = sum(len(v) for v in lists.values()) / (w.n_q_heads * w.n_blocks * (w.n_blocks + 1) / 2)
    _say(f"[parity] {w.name} tau={tau}: density {density:.4f}, all {len(every)} lists well formed")
    assert density < 0.1


@pytest.mark.slow
@pytest.mark.parametrize("name", ["qwen3-30b-a3b-128k-b64", "qwen3-30b-a3b-128k-b256"])
def test_qwen3_30b_128k_other_block_sizes_sampled(name):
    """The 128K layer at 64- and 256-token blocks; sampled rows."""
    w = WORKLOADS[name]
    M = w.n_blocks
    rows = H.sample_rows(w.n_q_heads, M, 16, seed=3, include=[(7, M - 1), (0, 1)])
    attn = H.sample_rows(w.n_q_heads, M, 4, seed=5, include=[(7, M - 1), (0, 1)])
    _full_check(w, select_rows=rows, attn_rows=attn)


@pytest.mark.slow
def test_qwen3_32b_64k_sampled():
    """64 query heads over 8 KV heads, two key-noise regimes; sampled rows."""
    w = WORKLOADS["qwen3-32b-64k"]
    M = w.n_blocks
    rows = H.sample_rows(w.n_q_heads, M, 24, seed=4, include=[(0, M - 1), (63, 300), (40, 2)])
    attn = H.sample_rows(w.n_q_heads, M, 5, seed=6, include=[(0, M - 1), (63, 300), (40, 2)])
    _full_check(w, select_rows=rows, attn_rows=attn)


@pytest.mark.slow
@pytest.mark.parametrize("layer", [0, 47])
def test_layer_schedule_layers_sampled(layer):
    """Layers of the 48-layer 128K sweep (per-layer key noise and needle
    counts); sampled rows."""
    from synth import layer_schedule
    w = layer_schedule(48)[layer]
    M = w.n_blocks
    rows = H.sample_rows(w.n_q_heads, M, 16, seed=10 + layer, include=[(3, M - 1), (30, 512)])
    _full_check(w, select_rows=rows, attn_rows=rows[:6])


def _fused_matches_two_calls(w: Workload, tau=None, forced=None, rows=None, attn_rows=None):
    """The fused entry point against the oracle (its own lists and O, as the
    two-call path is checked) and against rbs_select + rbs_sparse_prefill on
    the same inputs: lists, O and LSE bit for bit."""
    import torch
    import paper_2609_20971_amd as rbs
    r = _run(w, tau=tau, forced=forced)
    tb, tr = r["tau"]
    sink, local, recent = r["forced"]
    lse = torch.empty_like(r["lse"])
    counts, indices, O = rbs.rbs_select_attend(r["shape"], r["Qd"], r["Kd"], r["Vd"], r["stats"], tb, tr, sink,
                                               local, recent, 0.0, lse=lse)
    torch.cuda.synchronize()
    _oracle_check(w, r["inputs"], counts, indices, O, r["tau"], r["forced"], rows=rows, attn_rows=attn_rows,
                  label=f"fused {w.name} N={w.seq_len} B={w.block_size}")
    M = w.n_blocks
    assert torch.equal(counts, r["counts"])
    all_rows = [(h, i) for h in range(w.n_q_heads) for i in range(M)]
    assert H.gpu_rows(counts, indices, all_rows) == H.gpu_rows(r["counts"], r["indices"], all_rows)
    assert torch.equal(O.view(torch.int16), r["O"].view(torch.int16))
    assert torch.equal(lse, r["lse"])
    _say(f"[parity] fused {w.name} N={w.seq_len} B={w.block_size}: lists, O and LSE identical to the two calls")
    return r


@pytest.mark.parametrize("variant", [
    dict(),
    dict(seq_len=1000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=1),
    dict(seq_len=777, block_size=128, n_q_heads=2, n_kv_heads=2, seed=2),
    dict(seq_len=1300, block_size=256, n_q_heads=4, n_kv_heads=1, seed=3),
    dict(seq_len=5, block_size=128, n_q_heads=1, n_kv_heads=1, seed=5),
    dict(seq_len=8191, block_size=128, n_q_heads=8, n_kv_heads=2, seed=13),
])
def test_fused_select_attend_matches_two_calls(variant):
    w = WORKLOADS["tiny-2k"].with_(name="fused", **variant)
    M = w.n_blocks
    attn = None
    if M > 32:  # attention against the oracle on a sample of rows, the ragged last row included
        attn = H.sample_rows(w.n_q_heads, M, 16, seed=w.seed, include=[(0, M - 1), (w.n_q_heads - 1, M - 2)])
    _fused_matches_two_calls(w, attn_rows=attn)


def test_fused_select_attend_forced_and_dense_rows():
    w = WORKLOADS["tiny-2k"].with_(seq_len=1536, seed=7)
    _fused_matches_two_calls(w, tau=(0.0, 0.0), forced=(1, 2, 0))
    _fused_matches_two_calls(w, tau=(0.9, 0.95), forced=(0, 1, 2))


@pytest.mark.slow
def test_fused_select_attend_128k_matches_two_calls():
    """The headline layer through the fused entry point: sampled rows against
    the oracle, and identical to the two calls."""
    w = WORKLOADS["qwen3-30b-a3b-128k"]
    rows = H.sample_rows(w.n_q_heads, w.n_blocks, 24, seed=12, include=[(5, 1023), (31, 700), (0, 3)])
    _fused_matches_two_calls(w, rows=rows, attn_rows=rows[:10])


# ------------------------------------------------ supporting selectors (Table selector_ablation)

def _variant_check(w: Workload, variant: str, param: float, rows=None, inputs=None):
    """A supporting selector through the C ABI against the oracle's: box
    statistics to fp32 rounding, lists bit for bit outside the near-threshold
    band, the same structural invariants as the method's lists."""
    import torch
    import paper_2609_20971_amd as rbs
    if inputs is None:
        inputs = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Qd, Kd = H.to_device(inputs["q"]), H.to_device(inputs["k"])
    st = rbs.rbs_block_stats(shape, Kd)
    box = rbs.rbs_block_box(shape, Kd) if variant == "box" else None
    counts, indices = rbs.rbs_select_variant(shape, Qd, st, variant, param, w.n_sink, w.n_local, w.n_recent,
                                             box=box)
    torch.cuda.synchronize()
    Kf = f64_from_bf16_bits(inputs["k"])
    C, R = oracle.block_stats(Kf, w.block_size)
    Vc = Hw = None
    if variant == "box":
        Vc, Hw = oracle.block_box(Kf, w.block_size)
        for got, ref in ((box.center, Vc), (box.half, Hw)):
            g = got.double().cpu().numpy()
            assert np.abs(g - ref).max() <= 1e-6 * max(1.0, np.abs(ref).max())
    M = w.n_blocks
    rows = rows or [(h, i) for h in range(w.n_q_heads) for i in range(M)]
    Qf = f64_from_bf16_bits(inputs["q"])
    # The ABI takes the parameter as float32: the oracle gets that same value
    # (a budget of 0.3 is 0.30000001, whose ceil(rho n) can differ from 0.3's).
    param32 = float(np.float32(param))
    ref = oracle.select_variant(Qf, C, R, Vc, Hw, w.block_size, variant, param32, w.n_sink, w.n_local,
                                w.n_recent, rows=rows)
    lists = H.gpu_rows(counts, indices, rows)
    H.check_lists(lists, M, w.n_sink, w.n_local, w.n_recent)
    n_rows, compared, near = H.compare_masks(lists, ref)
    dens = sum(len(v) for v in lists.values()) / compared
    _say(f"[parity] selector {variant}({param}) {w.name} N={w.seq_len} B={w.block_size}: rows {n_rows} "
         f"blocks {compared} near-threshold flips {near}; density {dens:.4f}")
    return lists


@pytest.mark.parametrize("variant,param", [
    ("centroid", 0.9), ("centroid", 0.194), ("full_l2", 0.9), ("full_l2", 0.022), ("box", 0.0405), ("box", 0.3),
])
@pytest.mark.parametrize("shape", [
    dict(),
    dict(seq_len=1000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=1),
    dict(seq_len=777, block_size=128, n_q_heads=2, n_kv_heads=2, seed=2),
    dict(seq_len=1300, block_size=256, n_q_heads=4, n_kv_heads=1, seed=3),
])
def test_supporting_selectors_match_oracle(variant, param, shape):
    w = WORKLOADS["tiny-2k"].with_(name="selectors", **shape)
    _variant_check(w, variant, param)


def test_supporting_selector_extremes():
    """Threshold 0 keeps every causal block; a budget of 1 keeps every block."""
    w = WORKLOADS["tiny-2k"].with_(seq_len=1536, seed=7)
    for variant, param in (("centroid", 0.0), ("full_l2", 0.0), ("box", 1.0)):
        lists = _variant_check(w, variant, param)
        assert all(len(ids) == i + 1 for (h, i), ids in lists.items())


@pytest.mark.slow
@pytest.mark.parametrize("variant,param", [("centroid", 0.194), ("full_l2", 0.022), ("box", 0.0405)])
def test_supporting_selectors_32k_sampled(variant, param):
    w = WORKLOADS["qwen3-30b-a3b-32k"]
    rows = H.sample_rows(w.n_q_heads, w.n_blocks, 24, seed=8, include=[(3, w.n_blocks - 1)])
    _variant_check(w, variant, param, rows=rows)
