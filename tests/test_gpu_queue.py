"""GPU tests of the persistent attention launch (the work queues in the
attention workspace) against the one-workgroup-per-item launch.

Both launches run the same device code per (query head, query block) on the
same values, so the bar is bit equality of O and lse.  The oracle parity of
the attention itself is covered by the other GPU tests, which use the
persistent launch (the binding's default workspace)."""

from __future__ import annotations

import sys

import numpy as np
import pytest

from synth import WORKLOADS, batch_workloads, make_batch_inputs, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _setup(w, dense=False):
    import paper_2609_20971_amd as rbs
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    if dense:
        counts, indices = rbs.rbs_dense_indices(shape)
    else:
        st = rbs.rbs_block_stats(shape, K)
        counts, indices = rbs.rbs_select(shape, Q, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent)
    return shape, Q, K, V, counts, indices


def _attend(shape, Q, K, V, counts, indices, workspace, stream=None):
    import torch
    import paper_2609_20971_amd as rbs
    lse = torch.full((shape.n_q_heads, shape.n_tokens), 7.0, dtype=torch.float32, device=Q.device)
    O = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, lse=lse, stream=stream, workspace=workspace)
    return O, lse


def _assert_same(a, b, what):
    import torch
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]), f"{what}: O differs"
    assert torch.equal(a[1], b[1]), f"{what}: lse differs"


@pytest.mark.parametrize("B", [64, 128, 256])
@pytest.mark.parametrize("dense", [False, True])
def test_queue_launch_equals_one_workgroup_per_item(B, dense):
    w = WORKLOADS["tiny-2k"].with_(name="queue", seq_len=3000 if B < 256 else 2900, n_q_heads=8, n_kv_heads=2,
                                   block_size=B, seed=31 + B)
    _say(f"[queue] B={B} dense={dense} N={w.seq_len} Hq=8 Hkv=2")
    shape, Q, K, V, counts, indices = _setup(w, dense)
    grid = _attend(shape, Q, K, V, counts, indices, None)
    queued = _attend(shape, Q, K, V, counts, indices, "auto")
    _assert_same(grid, queued, f"B={B} dense={dense}")


def test_queue_with_fewer_items_than_queues():
    # One query block of two heads: 2 work items, 8 queues; six queues stay empty.
    w = WORKLOADS["tiny-2k"].with_(name="queue-tiny", seq_len=100, n_q_heads=2, n_kv_heads=1, block_size=128)
    _say("[queue] 2 items")
    shape, Q, K, V, counts, indices = _setup(w)
    _assert_same(_attend(shape, Q, K, V, counts, indices, None), _attend(shape, Q, K, V, counts, indices, "auto"),
                 "2 items")


def test_caller_workspace_with_stale_contents_and_reuse():
    """A caller's workspace holding arbitrary values is reset by the call; the
    same workspace then serves a second, smaller problem."""
    import torch
    ws = torch.randint(-2**31, 2**31 - 1, (64,), dtype=torch.int32, device="cuda")
    big = WORKLOADS["tiny-2k"].with_(name="queue-big", seq_len=4096, n_q_heads=4, n_kv_heads=2, block_size=128,
                                     seed=41)
    small = big.with_(name="queue-small", seq_len=700, seed=42)
    for w in (big, small):
        _say(f"[queue] caller workspace N={w.seq_len}")
        shape, Q, K, V, counts, indices = _setup(w)
        ref = _attend(shape, Q, K, V, counts, indices, None)
        got = _attend(shape, Q, K, V, counts, indices, ws)
        _assert_same(ref, got, f"N={w.seq_len}")
        ws.fill_(-5)  # stale, even negative, tickets before the next call


def test_queue_on_a_side_stream():
    import torch
    w = WORKLOADS["tiny-2k"].with_(name="queue-stream", seq_len=2500, n_q_heads=4, n_kv_heads=2, block_size=64,
                                   seed=43)
    _say("[queue] side stream")
    shape, Q, K, V, counts, indices = _setup(w)
    torch.cuda.synchronize()
    ref = _attend(shape, Q, K, V, counts, indices, None)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        got = _attend(shape, Q, K, V, counts, indices, "auto", stream=s)
    s.synchronize()
    _assert_same(ref, got, "side stream")


@pytest.mark.parametrize("B", [64, 128])
def test_queue_varlen_equals_one_workgroup_per_item(B):
    import torch
    import paper_2609_20971_amd as rbs
    base = WORKLOADS["tiny-2k"].with_(name="queue-varlen", n_q_heads=4, n_kv_heads=2, block_size=B)
    seqs = [700, 1536, 64, 2049, 1]
    _say(f"[queue] varlen B={B} seqs={seqs}")
    inputs = make_batch_inputs(batch_workloads(base, seqs, needles_per_2k=8))
    batch = rbs.Batch(seqs)
    shape = rbs.varlen_shape(batch, base.n_q_heads, base.n_kv_heads, B)
    Q, K, V = (H.to_device(inputs[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats_varlen(shape, batch, K)
    counts, indices = rbs.rbs_select_varlen(shape, batch, Q, st, base.tau_base, base.tau_rescue, base.n_sink,
                                            base.n_local, base.n_recent)
    out = []
    for ws in (None, "auto"):
        lse = torch.full((base.n_q_heads, batch.n_tokens), 7.0, dtype=torch.float32, device="cuda")
        O = rbs.rbs_sparse_prefill_varlen(shape, batch, Q, K, V, counts, indices, 0.0, lse=lse, workspace=ws)
        out.append((O, lse))
    _assert_same(out[0], out[1], f"varlen B={B}")


@pytest.mark.parametrize("B", [64, 128, 256])
def test_queue_fp8_equals_one_workgroup_per_item(B):
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="queue-fp8", seq_len=3000, n_q_heads=4, n_kv_heads=2, block_size=B,
                                   seed=44)
    _say(f"[queue] fp8 B={B}")
    shape, Q, K, V, counts, indices = _setup(w)
    f8 = rbs.rbs_fp8_prepare(shape, Q, K, V)
    out = []
    for ws in (None, "auto"):
        lse = torch.full((w.n_q_heads, w.seq_len), 7.0, dtype=torch.float32, device="cuda")
        O = rbs.rbs_sparse_prefill_fp8(shape, f8, counts, indices, lse=lse, workspace=ws)
        out.append((O, lse))
    _assert_same(out[0], out[1], "fp8")
    assert np.isfinite(out[1][1].cpu().numpy()).all()


@pytest.mark.parametrize("B", [64, 128])
def test_queue_fused_equals_one_workgroup_per_item(B):
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="queue-fused", seq_len=3000, n_q_heads=8, n_kv_heads=2, block_size=B,
                                   seed=45 + B)
    _say(f"[queue] fused B={B}")
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats(shape, K)
    out = []
    for ws in (None, "auto"):
        lse = torch.full((w.n_q_heads, w.seq_len), 7.0, dtype=torch.float32, device="cuda")
        counts, indices, O = rbs.rbs_select_attend(shape, Q, K, V, st, w.tau_base, w.tau_rescue, w.n_sink,
                                                   w.n_local, w.n_recent, lse=lse, workspace=ws)
        out.append((counts, indices, O, lse))
    torch.cuda.synchronize()
    assert torch.equal(out[0][0], out[1][0]), "counts"
    cnt = out[0][0].cpu().numpy()
    a, b = out[0][1].cpu().numpy(), out[1][1].cpu().numpy()
    for h in range(w.n_q_heads):
        for i in range(w.n_blocks):
            o = i * (i + 1) // 2
            assert np.array_equal(a[h, o:o + cnt[h, i]], b[h, o:o + cnt[h, i]]), (h, i)
    assert torch.equal(out[0][2], out[1][2]), "O"
    assert torch.equal(out[0][3], out[1][3]), "lse"


def test_persistent_attention_replays_from_a_graph():
    """The persistent launch captured in a graph (the queue reset is a kernel,
    not a memset): every replay equals the eager result, with eager calls on
    the same workspace between replays."""
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="queue-graph", seq_len=3000, n_q_heads=8, n_kv_heads=2, block_size=128,
                                   seed=47)
    _say("[queue] graph replays")
    shape, Q, K, V, counts, indices = _setup(w)
    ws = torch.empty(64, dtype=torch.int32, device="cuda")
    ref = _attend(shape, Q, K, V, counts, indices, ws)
    torch.cuda.synchronize()
    O = torch.empty_like(Q)
    lse = torch.empty((w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, O, lse=lse, workspace=ws)
    for rep in range(3):
        O.zero_()
        lse.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(O, ref[0]), f"replay {rep}: O differs"
        assert torch.equal(lse, ref[1]), f"replay {rep}: lse differs"
        eager = _attend(shape, Q, K, V, counts, indices, ws)  # the same workspace, between replays
        _assert_same(eager, ref, f"eager call after replay {rep}")
