"""GPU: the allocation-free attention entry point (rbs_sparse_prefill_noalloc)
against rbs_sparse_prefill on the same inputs and lists, through the C ABI:
two calls in a row on the library's static per-device scratch, the second on
a smaller input (the counters left by the first call must not leak into it),
O and LSE bit for bit; plus a graph-captured replay."""

from __future__ import annotations

import sys

import pytest

from synth import WORKLOADS, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _case(w, tau=(0.9, 0.95)):
    import torch
    import paper_2609_20971_amd as rbs
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats(shape, K)
    counts, indices = rbs.rbs_select(shape, Q, st, tau[0], tau[1], w.n_sink, w.n_local, w.n_recent)
    lse_ref = torch.empty((w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    O_ref = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, lse=lse_ref)
    torch.cuda.synchronize()
    return shape, Q, K, V, counts, indices, O_ref, lse_ref


def _noalloc(case):
    import torch
    import paper_2609_20971_amd as rbs
    shape, Q, K, V, counts, indices, _, lse_ref = case
    O = torch.full_like(Q, float("nan"))
    lse = torch.full_like(lse_ref, float("nan"))
    rbs.rbs_sparse_prefill_noalloc(shape, Q, K, V, counts, indices, O, lse=lse)
    torch.cuda.synchronize()
    return O, lse


def test_noalloc_matches_the_workspace_entry_point_twice_second_smaller():
    import torch
    big = WORKLOADS["tiny-2k"].with_(name="noalloc", seq_len=8191, block_size=128, n_q_heads=8, n_kv_heads=2,
                                     needles_per_kv_head=6, seed=41)
    small = WORKLOADS["tiny-2k"].with_(name="noalloc", seq_len=1000, block_size=64, n_q_heads=4, n_kv_heads=2,
                                       needles_per_kv_head=2, seed=42)
    for w in (big, small):
        _say(f"[noalloc] N={w.seq_len} Hq={w.n_q_heads} Hkv={w.n_kv_heads} B={w.block_size}")
        case = _case(w)
        O, lse = _noalloc(case)
        assert torch.equal(O.view(torch.int16), case[6].view(torch.int16))
        assert torch.equal(lse, case[7])
    _say("[noalloc] two calls in a row (second smaller): O and LSE identical to rbs_sparse_prefill")


def test_noalloc_graph_replay():
    """Captured in a HIP graph (no allocation inside the capture) and replayed
    three times with eager calls in between; every replay bit-identical."""
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="noalloc", seq_len=3000, needles_per_kv_head=4, seed=43)
    shape, Q, K, V, counts, indices, O_ref, lse_ref = case = _case(w)
    O = torch.empty_like(Q)
    lse = torch.empty_like(lse_ref)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        rbs.rbs_sparse_prefill_noalloc(shape, Q, K, V, counts, indices, O, lse=lse, stream=s)  # first call: lookup
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        rbs.rbs_sparse_prefill_noalloc(shape, Q, K, V, counts, indices, O, lse=lse, stream=s)
    for _ in range(3):
        O.zero_()
        lse.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(O.view(torch.int16), O_ref.view(torch.int16))
        assert torch.equal(lse, lse_ref)
        O2, lse2 = _noalloc(case)  # an eager call on the same scratch between replays
        assert torch.equal(O2.view(torch.int16), O_ref.view(torch.int16))
    _say("[noalloc] graph replays and eager calls in between: identical")
