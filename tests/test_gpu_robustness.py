"""GPU robustness: every output element is written, and nothing beyond the
outputs is.  Before each call the output buffers are poisoned (NaN, or
sentinel integers) and followed by canary words; afterwards every valid
element must have been overwritten, the list slots past each row's count must
be untouched (the ABI leaves them so), and every canary must be intact.  Both
attention launches (per item and persistent) are covered."""

from __future__ import annotations

import sys

import numpy as np
import pytest

from synth import WORKLOADS, batch_workloads, make_batch_inputs, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu

N_CANARY = 64
CANARY_I32 = -5
POISON_COUNT = -7
POISON_SLOT = -9
CANARY_F32 = 1.25e30


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _buffer(shape, dtype, poison, canary):
    """A poisoned tensor of `shape` followed by N_CANARY canary elements."""
    import torch
    n = int(np.prod(shape))
    full = torch.full((n + N_CANARY,), poison, dtype=dtype, device="cuda")
    full[n:] = canary
    return full, full[:n].view(*shape)


def _canary_intact(full, n, canary):
    import torch
    tail = full[n:]
    return bool(torch.all(tail == torch.tensor(canary, dtype=full.dtype, device=full.device)))


def _stats(rbs, shape):
    import torch
    M, hk, d = rbs.n_blocks(shape), shape.n_kv_heads, shape.head_dim
    bufs = {}
    for name, shp in (("centroids", (hk, M, d)), ("radii", (hk, M)), ("beta", (hk, M)), ("quantiles", (hk, 2))):
        bufs[name] = _buffer(shp, torch.float32, float("nan"), CANARY_F32)
    nsum = rbs.rbs_summary_bytes(shape)
    bufs["summary"] = _buffer((nsum,), torch.uint8, 0xAB, 0x5C)
    st = rbs.BlockStats(shape, *(bufs[k][1] for k in ("centroids", "radii", "beta", "quantiles", "summary")))
    return st, bufs


def _check_stats(bufs):
    import torch
    for name in ("centroids", "radii", "beta", "quantiles"):
        full, view = bufs[name]
        assert bool(torch.isfinite(view).all()), f"{name}: element not written"
        assert _canary_intact(full, view.numel(), CANARY_F32), f"{name}: written past its end"
    full, view = bufs["summary"]
    assert _canary_intact(full, view.numel(), 0x5C), "summary: written past its end"


def _check_lists(counts_buf, index_buf, Hq, M):
    import torch
    cfull, counts = counts_buf
    ifull, indices = index_buf
    assert _canary_intact(cfull, counts.numel(), CANARY_I32), "counts: written past its end"
    assert _canary_intact(ifull, indices.numel(), CANARY_I32), "indices: written past its end"
    cnt = counts.cpu().numpy()
    idx = indices.cpu().numpy()
    rows = np.arange(M)
    assert (cnt >= 1).all() and (cnt <= rows[None, :] + 1).all(), "a count outside [1, i + 1]"
    for h in range(Hq):
        for i in range(M):
            o, c = i * (i + 1) // 2, cnt[h, i]
            row = idx[h, o:o + i + 1]
            assert (np.diff(row[:c]) > 0).all() and row[c - 1] == i and row[0] >= 0, f"row {(h, i)} list"
            assert (row[c:] == POISON_SLOT).all(), f"row {(h, i)}: slots past the count were written"


def _check_attention(O_buf, lse_buf):
    import torch
    ofull, O = O_buf
    lfull, lse = lse_buf
    assert bool(torch.isfinite(O.float()).all()), "O: element not written"
    assert bool(torch.isfinite(lse).all()), "lse: element not written"
    assert _canary_intact(ofull, O.numel(), 7.0), "O: written past its end"
    assert _canary_intact(lfull, lse.numel(), CANARY_F32), "lse: written past its end"


CASES = [
    dict(seq_len=3000, n_q_heads=8, n_kv_heads=2, block_size=128, seed=61),   # ragged tail, GQA 4:1
    dict(seq_len=1000, n_q_heads=4, n_kv_heads=4, block_size=64, seed=62),    # no GQA
    dict(seq_len=2900, n_q_heads=4, n_kv_heads=1, block_size=256, seed=63),   # two softmax steps per block
    dict(seq_len=100, n_q_heads=2, n_kv_heads=1, block_size=128, seed=64),    # N < B
]


@pytest.mark.parametrize("workspace", [None, "auto"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"N{c['seq_len']}-B{c['block_size']}")
def test_outputs_fully_written_and_nothing_past_them(case, workspace):
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="robust", **case)
    _say(f"[robust] {case} workspace={workspace}")
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    M, Hq = w.n_blocks, w.n_q_heads
    st, sbufs = _stats(rbs, shape)
    rbs.rbs_block_stats(shape, K, st)
    cbuf = _buffer((Hq, M), torch.int32, POISON_COUNT, CANARY_I32)
    ibuf = _buffer((Hq, rbs.rbs_index_capacity(M)), torch.int32, POISON_SLOT, CANARY_I32)
    rbs.rbs_select(shape, Q, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent, cbuf[1], ibuf[1])
    obuf = _buffer((Hq, w.seq_len, 128), torch.bfloat16, float("nan"), 7.0)
    lbuf = _buffer((Hq, w.seq_len), torch.float32, float("nan"), CANARY_F32)
    rbs.rbs_sparse_prefill(shape, Q, K, V, cbuf[1], ibuf[1], 0.0, obuf[1], lse=lbuf[1], workspace=workspace)
    torch.cuda.synchronize()
    _check_stats(sbufs)
    _check_lists(cbuf, ibuf, Hq, M)
    _check_attention(obuf, lbuf)
    # The fused entry point into fresh poisoned buffers.
    cbuf = _buffer((Hq, M), torch.int32, POISON_COUNT, CANARY_I32)
    ibuf = _buffer((Hq, rbs.rbs_index_capacity(M)), torch.int32, POISON_SLOT, CANARY_I32)
    obuf = _buffer((Hq, w.seq_len, 128), torch.bfloat16, float("nan"), 7.0)
    lbuf = _buffer((Hq, w.seq_len), torch.float32, float("nan"), CANARY_F32)
    rbs.rbs_select_attend(shape, Q, K, V, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent, 0.0,
                          cbuf[1], ibuf[1], obuf[1], lse=lbuf[1], workspace=workspace)
    torch.cuda.synchronize()
    _check_lists(cbuf, ibuf, Hq, M)
    _check_attention(obuf, lbuf)


@pytest.mark.parametrize("workspace", [None, "auto"])
def test_varlen_outputs_fully_written_and_nothing_past_them(workspace):
    import torch
    import paper_2609_20971_amd as rbs
    base = WORKLOADS["tiny-2k"].with_(name="robust-varlen", n_q_heads=4, n_kv_heads=2, block_size=128)
    seqs = [700, 1536, 64, 2049, 1]
    _say(f"[robust] varlen {seqs} workspace={workspace}")
    inputs = make_batch_inputs(batch_workloads(base, seqs, needles_per_2k=8))
    batch = rbs.Batch(seqs)
    shape = rbs.varlen_shape(batch, base.n_q_heads, base.n_kv_heads, base.block_size)
    Q, K, V = (H.to_device(inputs[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats_varlen(shape, batch, K)
    Mt, Ct, T, Hq = rbs.rbs_varlen_blocks(shape, batch), rbs.rbs_varlen_index_capacity(shape, batch), sum(seqs), 4
    cbuf = _buffer((Hq, Mt), torch.int32, POISON_COUNT, CANARY_I32)
    ibuf = _buffer((Hq, Ct), torch.int32, POISON_SLOT, CANARY_I32)
    rbs.rbs_select_varlen(shape, batch, Q, st, base.tau_base, base.tau_rescue, base.n_sink, base.n_local,
                          base.n_recent, cbuf[1], ibuf[1])
    obuf = _buffer((Hq, T, 128), torch.bfloat16, float("nan"), 7.0)
    lbuf = _buffer((Hq, T), torch.float32, float("nan"), CANARY_F32)
    rbs.rbs_sparse_prefill_varlen(shape, batch, Q, K, V, cbuf[1], ibuf[1], 0.0, obuf[1], lse=lbuf[1],
                                  workspace=workspace)
    torch.cuda.synchronize()
    assert _canary_intact(cbuf[0], cbuf[1].numel(), CANARY_I32)
    assert _canary_intact(ibuf[0], ibuf[1].numel(), CANARY_I32)
    assert bool((cbuf[1] >= 1).all())
    _check_attention(obuf, lbuf)


@pytest.mark.parametrize("B", [64, 128, 256])
def test_fp8_outputs_fully_written_and_nothing_past_them(B):
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="robust-fp8", seq_len=1500, n_q_heads=4, n_kv_heads=2, block_size=B,
                                   seed=65)
    _say(f"[robust] fp8 B={B}")
    inp = make_inputs(w)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Q, K, V = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats(shape, K)
    counts, indices = rbs.rbs_select(shape, Q, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent)
    amax = _buffer((w.n_q_heads + 2 * w.n_kv_heads,), torch.float32, float("nan"), CANARY_F32)
    q8 = _buffer((w.n_q_heads, w.seq_len, 128), torch.uint8, 0xFF, 0x5C)
    k8 = _buffer((w.n_kv_heads, w.seq_len, 128), torch.uint8, 0xFF, 0x5C)
    vt = _buffer((rbs.rbs_fp8_vt_bytes(shape),), torch.uint8, 0xFF, 0x5C)
    f8 = rbs.Fp8Inputs(amax[1], q8[1], k8[1], vt[1])
    rbs.rbs_fp8_amax(shape, Q, K, V, f8.amax)
    rbs.rbs_fp8_pack(shape, Q, K, V, f8)
    obuf = _buffer((w.n_q_heads, w.seq_len, 128), torch.bfloat16, float("nan"), 7.0)
    lbuf = _buffer((w.n_q_heads, w.seq_len), torch.float32, float("nan"), CANARY_F32)
    rbs.rbs_sparse_prefill_fp8(shape, f8, counts, indices, O=obuf[1], lse=lbuf[1])
    torch.cuda.synchronize()
    assert bool(torch.isfinite(amax[1]).all()) and _canary_intact(amax[0], amax[1].numel(), CANARY_F32)
    for buf in (q8, k8, vt):
        assert _canary_intact(buf[0], buf[1].numel(), 0x5C), "FP8 copy written past its end"
    # 0xFF is E4M3's NaN code: after packing no code may be NaN (finite inputs saturate).
    for buf in (q8, k8, vt):
        assert not bool((buf[1] == 0xFF).any()) and not bool((buf[1] == 0x7F).any()), "a code not written"
    _check_attention(obuf, lbuf)
