"""GPU parity of the varlen (batched) calls: a batch of independent sequences
packed along the token axis, each processed as on its own.

Two bars: the float64 oracle run on every sequence alone (stats, masks under
the usual parity rules, attention on the GPU's own lists), and the
single-sequence calls of the library on each sequence, which the batched
launch must reproduce bit for bit (the same device code on the same values)."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, batch_workloads, f64_from_bf16_bits, make_batch_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu

MIXED = [700, 1536, 64, 2049, 1]   # ragged tails, a one-block and a one-token sequence


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _base(B, **kw):
    return WORKLOADS["tiny-2k"].with_(name="varlen", n_q_heads=4, n_kv_heads=2, block_size=B, **kw)


def _run_varlen(base, seq_tokens, inputs=None, dense=False):
    import torch
    import paper_2609_20971_amd as rbs
    if inputs is None:
        inputs = make_batch_inputs(batch_workloads(base, seq_tokens, needles_per_2k=8))
    batch = rbs.Batch(seq_tokens)
    shape = rbs.varlen_shape(batch, base.n_q_heads, base.n_kv_heads, base.block_size)
    Qd, Kd, Vd = (H.to_device(inputs[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats_varlen(shape, batch, Kd)
    if dense:
        counts, indices = rbs.rbs_dense_indices_varlen(shape, batch)
    else:
        counts, indices = rbs.rbs_select_varlen(shape, batch, Qd, st, base.tau_base, base.tau_rescue,
                                                base.n_sink, base.n_local, base.n_recent)
    lse = torch.empty((base.n_q_heads, batch.n_tokens), dtype=torch.float32, device="cuda")
    O = rbs.rbs_sparse_prefill_varlen(shape, batch, Qd, Kd, Vd, counts, indices, 0.0, lse=lse)
    torch.cuda.synchronize()
    return dict(batch=batch, inputs=inputs, Qd=Qd, Kd=Kd, Vd=Vd, stats=st, counts=counts, indices=indices, O=O,
                lse=lse)


def _seq_views(r, base):
    """Per sequence: (token range, block range, list-slot range)."""
    B = base.block_size
    tok, blk, cap = [0], [0], [0]
    for n in r["batch"].seq_tokens:
        m = -(-n // B)
        tok.append(tok[-1] + n)
        blk.append(blk[-1] + m)
        cap.append(cap[-1] + m * (m + 1) // 2)
    return tok, blk, cap


def _seq_lists(r, base, s, rows):
    """{(h, i): ids} of sequence s from the batched counts/indices."""
    tok, blk, cap = _seq_views(r, base)
    cnt = r["counts"].cpu().numpy()[:, blk[s]:blk[s + 1]]
    idx = r["indices"].cpu().numpy()[:, cap[s]:cap[s + 1]]
    return {(h, i): idx[h, i * (i + 1) // 2:i * (i + 1) // 2 + cnt[h, i]].tolist() for (h, i) in rows}


@pytest.mark.parametrize("B", [64, 128, 256])
def test_varlen_matches_the_oracle_per_sequence(B):
    base = _base(B)
    _say(f"[varlen] oracle parity B={B} seqs={MIXED}")
    r = _run_varlen(base, MIXED)
    inp = r["inputs"]
    Qf, Kf, Vf = (f64_from_bf16_bits(inp[x]) for x in ("q", "k", "v"))
    C, R, beta, rq = oracle.batch_block_stats(Kf, MIXED, B)
    rep = H.check_stats(r["stats"], C, R, beta, rq)
    ref = oracle.batch_select(Qf, Kf, MIXED, B, base.tau_base, base.tau_rescue, base.n_sink, base.n_local,
                              base.n_recent)
    Qs, Ks, Vs = (oracle.batch_sequences(X, MIXED) for X in (Qf, Kf, Vf))
    tok, _, _ = _seq_views(r, base)
    Og = H.bf16_tensor_to_f64(r["O"])
    near_total, worst = 0, 0.0
    for s, n in enumerate(MIXED):
        M = -(-n // B)
        rows = [(h, i) for h in range(base.n_q_heads) for i in range(M)]
        lists = _seq_lists(r, base, s, rows)
        H.check_lists(lists, M, base.n_sink, base.n_local, base.n_recent)
        _, _, near = H.compare_masks(lists, ref[s])
        near_total += near
        err = H.max_abs_attention_error(Og[:, tok[s]:tok[s + 1]], Qs[s], Ks[s], Vs[s], base.group, B, lists, n)
        worst = max(worst, err)
    _say(f"[varlen] B={B}: stats {rep}; near-threshold flips {near_total}; attention max-abs {worst:.3e}")
    assert worst <= H.ATTN_ATOL


def _single_calls(r, base, s):
    """The single-sequence calls on sequence s alone (contiguous copies)."""
    import torch
    import paper_2609_20971_amd as rbs
    tok, _, _ = _seq_views(r, base)
    n = r["batch"].seq_tokens[s]
    Q, K, V = (r[x][:, tok[s]:tok[s + 1]].contiguous() for x in ("Qd", "Kd", "Vd"))
    shape = rbs.make_shape(n, base.n_q_heads, base.n_kv_heads, base.block_size)
    st = rbs.rbs_block_stats(shape, K)
    counts, indices = rbs.rbs_select(shape, Q, st, base.tau_base, base.tau_rescue, base.n_sink, base.n_local,
                                     base.n_recent)
    lse = torch.empty((base.n_q_heads, n), dtype=torch.float32, device="cuda")
    O = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, lse=lse)
    return st, counts, indices, O, lse


def _assert_bitwise_equal_to_single_calls(r, base):
    import torch
    tok, blk, cap = _seq_views(r, base)
    for s in range(len(r["batch"].seq_tokens)):
        st, counts, indices, O, lse = _single_calls(r, base, s)
        torch.cuda.synchronize()
        b0, b1 = blk[s], blk[s + 1]
        assert torch.equal(r["stats"].centroids[:, b0:b1], st.centroids), f"seq {s} centroids"
        assert torch.equal(r["stats"].radii[:, b0:b1], st.radii), f"seq {s} radii"
        assert torch.equal(r["stats"].beta[:, b0:b1], st.beta), f"seq {s} beta"
        assert torch.equal(r["stats"].quantiles[s], st.quantiles), f"seq {s} quantiles"
        assert torch.equal(r["counts"][:, b0:b1], counts), f"seq {s} counts"
        # Compare only the filled slots of every row.
        M = b1 - b0
        vi = r["indices"][:, cap[s]:cap[s + 1]]
        cnt = counts.cpu().numpy()
        a, b = vi.cpu().numpy(), indices.cpu().numpy()
        for i in range(M):
            o = i * (i + 1) // 2
            for h in range(base.n_q_heads):
                c = cnt[h, i]
                assert np.array_equal(a[h, o:o + c], b[h, o:o + c]), f"seq {s} row {(h, i)}"
        assert torch.equal(r["O"][:, tok[s]:tok[s + 1]], O), f"seq {s} O"
        assert torch.equal(r["lse"][:, tok[s]:tok[s + 1]], lse), f"seq {s} lse"


@pytest.mark.parametrize("B", [64, 128, 256])
def test_varlen_equals_single_sequence_calls(B):
    base = _base(B)
    _say(f"[varlen] bitwise vs single calls B={B} seqs={MIXED}")
    _assert_bitwise_equal_to_single_calls(_run_varlen(base, MIXED), base)


def test_varlen_dense_lists():
    import torch
    import paper_2609_20971_amd as rbs
    base = _base(128)
    _say(f"[varlen] dense lists seqs={MIXED}")
    r = _run_varlen(base, MIXED, dense=True)
    tok, blk, cap = _seq_views(r, base)
    for s, n in enumerate(MIXED):
        M = blk[s + 1] - blk[s]
        assert (r["counts"][:, blk[s]:blk[s + 1]].cpu().numpy() == np.arange(1, M + 1)[None]).all()
        shape = rbs.make_shape(n, base.n_q_heads, base.n_kv_heads, base.block_size)
        Q, K, V = (r[x][:, tok[s]:tok[s + 1]].contiguous() for x in ("Qd", "Kd", "Vd"))
        counts, indices = rbs.rbs_dense_indices(shape)
        O = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices)
        torch.cuda.synchronize()
        assert torch.equal(r["O"][:, tok[s]:tok[s + 1]], O), f"seq {s}"
    # Full selection is dense causal attention of each sequence alone.
    inp = r["inputs"]
    Qf, Kf, Vf = (f64_from_bf16_bits(inp[x]) for x in ("q", "k", "v"))
    Og = H.bf16_tensor_to_f64(r["O"])
    for s, (Qs, Ks, Vs) in enumerate(zip(*(oracle.batch_sequences(X, MIXED) for X in (Qf, Kf, Vf)))):
        if MIXED[s] > 1600:
            continue  # the O(N^2) brute force on the two short ones and the mid one is enough
        ref = oracle.dense_causal_attention(Qs[3], Ks[1], Vs[1])
        assert np.abs(Og[3, tok[s]:tok[s + 1]] - ref).max() <= H.ATTN_ATOL


def test_varlen_sixty_four_sequences():
    rng = np.random.default_rng(5)
    seqs = [int(x) for x in rng.integers(1, 400, size=64)]
    seqs[7], seqs[40] = 1, 64
    base = _base(64)
    _say(f"[varlen] 64 sequences, {sum(seqs)} tokens")
    _assert_bitwise_equal_to_single_calls(_run_varlen(base, seqs), base)


@pytest.mark.slow
def test_varlen_qwen3_batch_of_four_32k():
    """The paper's batch-four setting at 32K per prompt: Qwen3-30B-A3B-shaped
    sequences, bitwise equal to four single-sequence runs."""
    base = WORKLOADS["qwen3-30b-a3b-32k"]
    seqs = [32768] * 4
    _say(f"[varlen] qwen3-30b-a3b 4 x 32K")
    _assert_bitwise_equal_to_single_calls(_run_varlen(base, seqs, inputs=make_batch_inputs(
        batch_workloads(base, seqs))), base)
