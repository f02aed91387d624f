"""GPU: the boundary's strides and externally held statistics.

Q, K and V as a serving stack holds them -- token-major [N][H][d], or slices of
one fused QKV buffer [N][H_q + 2 H_kv][d] -- passed as (head, token, dim)
views with the strides in rbs_shape: every stage must read them and write O
in Q's layout, with results identical bit for bit to the dense [H][N][d]
layout, and the lists and O checked against the oracle.  rbs_stats_summarize
must rebuild the select-ready summary that rbs_block_stats writes, and select
from statistics the oracle computed."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, f64_from_bf16_bits, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _token_major(x):
    """A (head, token, dim) view of a new token-major [N][H][d] copy of x."""
    return x.transpose(0, 1).contiguous().transpose(0, 1)


def _fused_qkv(Q, K, V):
    """(head, token, dim) views of one token-major [N][H_q + 2 H_kv][d] buffer."""
    import torch
    hq, hk = Q.shape[0], K.shape[0]
    buf = torch.cat([Q.transpose(0, 1), K.transpose(0, 1), V.transpose(0, 1)], dim=1).contiguous()
    return (buf[:, :hq].transpose(0, 1), buf[:, hq:hq + hk].transpose(0, 1),
            buf[:, hq + hk:].transpose(0, 1))


def _path(rbs, shape, Q, K, V, w, torch, fused=False):
    st = rbs.rbs_block_stats(shape, K)
    lse = torch.empty((w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    if fused:
        counts, indices, O = rbs.rbs_select_attend(shape, Q, K, V, st, w.tau_base, w.tau_rescue, w.n_sink,
                                                   w.n_local, w.n_recent, 0.0, lse=lse)
    else:
        counts, indices = rbs.rbs_select(shape, Q, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local, w.n_recent)
        O = rbs.rbs_sparse_prefill(shape, Q, K, V, counts, indices, 0.0, lse=lse)
    torch.cuda.synchronize()
    return st, counts, indices, O, lse


@pytest.mark.parametrize("layout", ["token_major", "fused_qkv"])
@pytest.mark.parametrize("variant", [
    dict(),
    dict(seq_len=1000, block_size=64, n_q_heads=4, n_kv_heads=2, seed=1),
    dict(seq_len=1300, block_size=256, n_q_heads=4, n_kv_heads=1, seed=3),
])
def test_strided_inputs_match_dense_layout_and_oracle(layout, variant):
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(name="layout", needles_per_kv_head=4, **variant)
    _say(f"[layout] {layout} N={w.seq_len} Hq={w.n_q_heads} Hkv={w.n_kv_heads} B={w.block_size}")
    inp = make_inputs(w)
    Qd, Kd, Vd = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    if layout == "token_major":
        Qs, Ks, Vs = _token_major(Qd), _token_major(Kd), _token_major(Vd)
    else:
        Qs, Ks, Vs = _fused_qkv(Qd, Kd, Vd)
    # Really strided: heads adjacent within a token (a single head's view is the dense layout anyway).
    assert Qs.stride(0) == 128 and (w.n_kv_heads == 1 or Ks.stride(0) == 128)
    for fused in (False, True):
        ref = _path(rbs, shape, Qd, Kd, Vd, w, torch, fused)
        got = _path(rbs, shape, Qs, Ks, Vs, w, torch, fused)
        for a in ("centroids", "radii", "beta", "quantiles"):
            assert torch.equal(getattr(ref[0], a), getattr(got[0], a)), a
        assert H.summaries_equal(ref[0].summary, got[0].summary, w.n_kv_heads, w.n_blocks)
        assert torch.equal(ref[1], got[1])
        M = w.n_blocks
        rows = [(h, i) for h in range(w.n_q_heads) for i in range(M)]
        assert H.gpu_rows(ref[1], ref[2], rows) == H.gpu_rows(got[1], got[2], rows)
        assert got[3].stride() == Qs.stride()
        assert torch.equal(ref[3].view(torch.int16), got[3].contiguous().view(torch.int16))
        assert torch.equal(ref[4], got[4])
    # And against the oracle, from the strided run's own outputs.
    Kf = f64_from_bf16_bits(inp["k"])
    C, R = oracle.block_stats(Kf, w.block_size)
    beta, rq = oracle.rescue_coefficients(R)
    H.check_stats(got[0], C, R, beta, rq)
    Qf = f64_from_bf16_bits(inp["q"])
    ref_rows = oracle.select(Qf, C, R, beta, w.block_size, w.tau_base, w.tau_rescue, w.n_sink, w.n_local,
                             w.n_recent, rows=rows)
    lists = H.gpu_rows(got[1], got[2], rows)
    H.check_lists(lists, M, w.n_sink, w.n_local, w.n_recent)
    _, compared, near = H.compare_masks(lists, ref_rows)
    Og = H.bf16_tensor_to_f64(got[3].contiguous())
    err = H.max_abs_attention_error(Og, Qf, Kf, f64_from_bf16_bits(inp["v"]), w.group, w.block_size, lists,
                                    w.seq_len)
    _say(f"[layout] {layout}: identical to the dense layout (two calls and fused); oracle: {compared} blocks, "
         f"{near} near-threshold flips, attention max-abs {err:.3e}")
    assert err <= H.ATTN_ATOL


def test_strided_fp8_and_varlen_match_dense_layout():
    import torch
    import paper_2609_20971_amd as rbs
    from synth import batch_workloads, make_batch_inputs
    w = WORKLOADS["tiny-2k"].with_(name="layout", seq_len=1536, needles_per_kv_head=4, seed=21)
    inp = make_inputs(w)
    Qd, Kd, Vd = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    Qs, Ks, Vs = _fused_qkv(Qd, Kd, Vd)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    counts, indices = rbs.rbs_dense_indices(shape)
    f8d = rbs.rbs_fp8_prepare(shape, Qd, Kd, Vd)
    f8s = rbs.rbs_fp8_prepare(shape, Qs, Ks, Vs)
    Od = rbs.rbs_sparse_prefill_fp8(shape, f8d, counts, indices)
    Os = torch.empty_strided(tuple(Qs.shape), Qs.stride(), dtype=torch.bfloat16, device="cuda")
    rbs.rbs_sparse_prefill_fp8(shape, f8s, counts, indices, O=Os)
    torch.cuda.synchronize()
    for name in ("amax", "Q8", "K8", "V8t"):
        assert torch.equal(getattr(f8d, name), getattr(f8s, name)), name
    assert torch.equal(Od.view(torch.int16), Os.contiguous().view(torch.int16))
    _say("[layout] FP8 packing and attention from a fused QKV buffer: identical to the dense layout")

    lens = [700, 1536, 64, 129]
    ws = batch_workloads(WORKLOADS["tiny-2k"].with_(name="layout-batch"), lens)
    binp = make_batch_inputs(ws)
    batch = rbs.Batch(lens)
    vshape = rbs.varlen_shape(batch, w.n_q_heads, w.n_kv_heads, w.block_size)
    Qd, Kd, Vd = (H.to_device(binp[x]) for x in ("q", "k", "v"))
    Qs, Ks, Vs = _fused_qkv(Qd, Kd, Vd)
    out = []
    for Q, K, V in ((Qd, Kd, Vd), (Qs, Ks, Vs)):
        st = rbs.rbs_block_stats_varlen(vshape, batch, K)
        c, ix = rbs.rbs_select_varlen(vshape, batch, Q, st, w.tau_base, w.tau_rescue, w.n_sink, w.n_local,
                                      w.n_recent)
        O = rbs.rbs_sparse_prefill_varlen(vshape, batch, Q, K, V, c, ix)
        torch.cuda.synchronize()
        out.append((st.summary, c, ix, O.contiguous()))
    (s0, c0, i0, o0), (s1, c1, i1, o1) = out
    m_tot = rbs.rbs_varlen_blocks(vshape, batch)
    assert H.summaries_equal(s0, s1, w.n_kv_heads, m_tot) and torch.equal(c0, c1)
    for h in range(w.n_q_heads):  # list slots past the counts are not written; compare the written ones
        assert torch.equal(c0[h], c1[h])
    cap = rbs.rbs_varlen_index_capacity(vshape, batch)
    mask = torch.zeros_like(i0, dtype=torch.bool)
    cnt = c0.cpu().numpy()
    tab = np.cumsum([0] + [rbs.n_blocks(rbs.make_shape(n, 1, 1, w.block_size)) for n in lens])
    capo = np.cumsum([0] + [m * (m + 1) // 2 for m in np.diff(tab)])
    for h in range(w.n_q_heads):
        for s_ in range(len(lens)):
            for i in range(tab[s_ + 1] - tab[s_]):
                base = capo[s_] + i * (i + 1) // 2
                mask[h, base:base + cnt[h, tab[s_] + i]] = True
    assert i0.shape[1] == cap
    assert torch.equal(i0[mask], i1[mask])
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))
    _say("[layout] varlen batch from a fused QKV buffer: identical to the dense layout")


def test_stats_summarize_rebuilds_the_summary():
    """rbs_stats_summarize from the fp32 statistics rebuilds, bit for bit, the
    select-ready summary that rbs_block_stats writes (Sec. 3.1)."""
    import torch
    import paper_2609_20971_amd as rbs
    for variant in (dict(), dict(seq_len=1300, block_size=256, n_q_heads=4, n_kv_heads=1, seed=3)):
        w = WORKLOADS["tiny-2k"].with_(**variant)
        inp = make_inputs(w)
        shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
        st = rbs.rbs_block_stats(shape, H.to_device(inp["k"]))
        again = rbs.BlockStats(shape, st.centroids.clone(), st.radii.clone(), st.beta.clone(),
                               st.quantiles.clone(), torch.full_like(st.summary, 0xCD))
        rbs.rbs_stats_summarize(shape, again)
        torch.cuda.synchronize()
        assert H.summaries_equal(again.summary, st.summary, w.n_kv_heads, w.n_blocks)


def test_selection_from_oracle_statistics():
    """Statistics computed elsewhere (here: the oracle's, rounded to fp32) go
    through rbs_stats_summarize into rbs_select; the lists match the oracle's
    selection on the same statistics outside the near-threshold band."""
    import torch
    import paper_2609_20971_amd as rbs
    w = WORKLOADS["tiny-2k"].with_(seq_len=1536, seed=33)
    inp = make_inputs(w)
    Kf = f64_from_bf16_bits(inp["k"])
    C, R = oracle.block_stats(Kf, w.block_size)
    beta, rq = oracle.rescue_coefficients(R)
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    dev = dict(dtype=torch.float32, device="cuda")
    st = rbs.BlockStats(shape, torch.tensor(C, **dev), torch.tensor(R, **dev), torch.tensor(beta, **dev),
                        torch.tensor(rq, **dev), torch.empty(rbs.rbs_summary_bytes(shape), dtype=torch.uint8,
                                                             device="cuda"))
    rbs.rbs_stats_summarize(shape, st)
    counts, indices = rbs.rbs_select(shape, H.to_device(inp["q"]), st, w.tau_base, w.tau_rescue, w.n_sink,
                                     w.n_local, w.n_recent)
    torch.cuda.synchronize()
    M = w.n_blocks
    rows = [(h, i) for h in range(w.n_q_heads) for i in range(M)]
    ref = oracle.select(f64_from_bf16_bits(inp["q"]), C, R, beta, w.block_size, w.tau_base, w.tau_rescue, w.n_sink,
                        w.n_local, w.n_recent, rows=rows)
    lists = H.gpu_rows(counts, indices, rows)
    H.check_lists(lists, M, w.n_sink, w.n_local, w.n_recent)
    _, compared, near = H.compare_masks(lists, ref)
    _say(f"[layout] selection from oracle statistics: {compared} blocks, {near} near-threshold flips")
