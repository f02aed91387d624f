"""Debug mode on the GPU (rbs_set_debug): every call drains its stream, the
results are those of the normal mode bit for bit, and a Q that the selector's
f16 operands cannot hold (an element of magnitude 65536 or more, or not
finite) is refused with RBS_ERR_RANGE before anything is written."""

from __future__ import annotations

import sys

import numpy as np
import pytest

from synth import WORKLOADS, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _calls(rbs, w, Q, K, V):
    """Stats, selection, attention and the fused call; returns their outputs."""
    import torch
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    stats = rbs.BlockStats.allocate(shape, Q.device)
    rbs.rbs_block_stats(shape, K, stats)
    counts, indices = rbs.allocate_lists(shape, Q.device)
    counts.fill_(-7)
    rbs.rbs_select(shape, Q, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent, counts, indices)
    O = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices)
    fc, fi = rbs.allocate_lists(shape, Q.device)
    _, _, Of = rbs.rbs_select_attend(shape, Q, K, V, stats, w.tau_base, w.tau_rescue, w.n_sink, w.n_local,
                                      w.n_recent, 0.0, fc, fi)
    torch.cuda.synchronize()
    return counts, indices, O, fc, fi, Of, stats, shape


def test_debug_mode_matches_normal_mode_and_rejects_out_of_range_queries():
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(seq_len=1000, seed=41)
    _say(f"[debug] N={w.seq_len} B={w.block_size}")
    inp = make_inputs(w)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    base = _calls(rbs, w, Q, K, V)
    prev = rbs.rbs_set_debug(True)
    try:
        dbg = _calls(rbs, w, Q, K, V)
        for a, b in zip(base[:6], dbg[:6]):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b)
        stats, shape = dbg[6], dbg[7]
        # 65280, the largest bf16 below f16's 65504, passes; 65536 and NaN do not.
        for bits, ok in ((0x477F, True), (0x4780, False), (0xC780, False), (0x7FC0, False)):
            qb = inp["q"].copy()
            qb[1, 517, 33] = bits
            Qb = H.to_device(qb)
            counts, indices = rbs.allocate_lists(shape, Q.device)
            counts.fill_(-7)
            args = (w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent)
            if ok:
                rbs.rbs_select(shape, Qb, stats, *args, counts, indices)
                assert (counts.cpu().numpy() > 0).all()
                continue
            with pytest.raises(rbs.RbsError) as e:
                rbs.rbs_select(shape, Qb, stats, *args, counts, indices)
            assert e.value.status == rbs.RBS_ERR_RANGE
            with pytest.raises(rbs.RbsError) as e:
                rbs.rbs_select_attend(shape, Qb, K, V, stats, *args, 0.0, counts, indices)
            assert e.value.status == rbs.RBS_ERR_RANGE
            torch.cuda.synchronize()
            assert (counts.cpu().numpy() == -7).all(), "nothing is written when the range check fails"
    finally:
        rbs.rbs_set_debug(prev)
    assert rbs.rbs_set_debug(prev) == prev
