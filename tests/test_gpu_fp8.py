"""GPU parity of the FP8-input attention (rbs_fp8_amax, rbs_fp8_pack,
rbs_sparse_prefill_fp8) against the float64 oracle.

* amax and the E4M3 codes of Q, K and V: bit-exact against the oracle's own
  quantisation of the same bf16 inputs (integer work);
* attention: the oracle's attention_on_mask on the dequantised inputs and the
  GPU's own lists, within a bound derived from the arithmetic (per output
  element, see _bound): P is rounded to E4M3 (unit roundoff u = 2^-4), the FP8
  matrix core accumulates with a relative error below 2^-7 of the sum of
  magnitudes (probe: at most 2^-9 observed), O is rounded to bf16.  The
  kernel scales P so that the row's reference maximum (at most 2 binades
  below the true maximum) sits at 2^6; a term more than 12 binades below the
  maximum may fall into E4M3's subnormal range, where the rounding error is
  absolute (at most 2^-10, i.e. 2^-16 of the largest term)."""

from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, Workload, f64_from_bf16_bits, make_inputs
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu

U8 = 2.0 ** -4         # unit roundoff of E4M3 (3 mantissa bits, round to nearest)
ACC = 2.0 ** -7        # allowance for the FP8 matrix core's accumulation error (relative to sum of |terms|)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _vt_key(p: int) -> int:
    """Key held at position p of a V^T tile row (the kernel's documented order)."""
    s, g, b = p >> 6, (p >> 5) & 1, p & 31
    r = b & 15
    return 64 * s + 32 * (b >> 4) + 8 * (r >> 2) + 4 * g + (r & 3)


def _vt_layout(T: np.ndarray, B: int) -> np.ndarray:
    """Bytes of one block's V^T tile from its [d][position] matrix T, in the
    documented layout: row-major [d][B], or for B = 256 two [d][128] halves."""
    if B <= 128:
        return T.reshape(-1)
    return np.concatenate([T[:, :128].reshape(-1), T[:, 128:].reshape(-1)])


def _run(w: Workload, tau=None, forced=None):
    import torch
    import paper_2609_20971_amd as rbs
    inp = make_inputs(w)
    tb, tr = (w.tau_base, w.tau_rescue) if tau is None else tau
    sink, local, recent = (w.n_sink, w.n_local, w.n_recent) if forced is None else forced
    shape = rbs.make_shape(w.seq_len, w.n_q_heads, w.n_kv_heads, w.block_size)
    Qd, Kd, Vd = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    st = rbs.rbs_block_stats(shape, Kd)
    counts, indices = rbs.rbs_select(shape, Qd, st, tb, tr, sink, local, recent)
    f8 = rbs.rbs_fp8_prepare(shape, Qd, Kd, Vd)
    lse = torch.empty((w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    O = rbs.rbs_sparse_prefill_fp8(shape, f8, counts, indices, lse=lse)
    torch.cuda.synchronize()
    return dict(inp=inp, f8=f8, counts=counts, indices=indices, O=O, lse=lse)


def _oracle_fp8(inp):
    """The oracle's own quantisation of the bf16 inputs: codes, scales, values."""
    out = {}
    for x in ("q", "k", "v"):
        X = f64_from_bf16_bits(inp[x])
        amax = oracle.fp8_amax(X)
        codes, deq = oracle.fp8_quantize(X, amax)
        out[x] = (amax, codes, deq, oracle.fp8_dequantize(codes, deq))
    return out


def _check_pack(r, ref, w):
    f8 = r["f8"]
    amax = f8.amax.cpu().numpy().astype(np.float64)
    Hq, Hkv, N, B = w.n_q_heads, w.n_kv_heads, w.seq_len, w.block_size
    assert np.array_equal(amax[:Hq], ref["q"][0]) and np.array_equal(amax[Hq:Hq + Hkv], ref["k"][0])
    assert np.array_equal(amax[Hq + Hkv:], ref["v"][0])
    assert np.array_equal(f8.Q8.cpu().numpy(), ref["q"][1]), "Q codes"
    assert np.array_equal(f8.K8.cpu().numpy(), ref["k"][1]), "K codes"
    M = w.n_blocks
    vt = f8.V8t.cpu().numpy().reshape(Hkv, M, 128 * B)
    keys = np.array([_vt_key(p) for p in range(B)])
    assert np.array_equal(np.sort(keys), np.arange(B))  # a permutation of the block's keys
    vcodes = ref["v"][1]
    for g in range(Hkv):
        for b in range(M):
            want = np.zeros((B, 128), dtype=np.uint8)
            n = min(B, N - b * B)
            want[:n] = vcodes[g, b * B:b * B + n]
            assert np.array_equal(vt[g, b], _vt_layout(want[keys].T, B)), f"V^T tile ({g}, {b})"


def _bound(Qh, Kg, Vg, B, i, ids, O_ref, scale):
    """Per-element tolerance of one query block (derivation in the module doc):
    (2u/(1-u) + 2(e^{2 D} - 1)) * sum_j w_j |v_j - O| + ACC (sum_j w_j |v_j| + |O|)
    + 2^-8 |O|, where D = ACC * max_j sum_k |q_k k_jk| * scale bounds the logit
    error of the matrix core's accumulation."""
    N, d = Kg.shape
    s, e = i * B, min((i + 1) * B, N)
    key_pos = np.concatenate([np.arange(b * B, min((b + 1) * B, N)) for b in sorted(ids)])
    Kr, Vr = Kg[key_pos], Vg[key_pos]
    q = Qh[s:e]
    logits = (q @ Kr.T) * scale
    causal = key_pos[None, :] <= np.arange(s, e)[:, None]
    logits = np.where(causal, logits, -np.inf)
    wts = np.exp(logits - logits.max(axis=1, keepdims=True))
    wts /= wts.sum(axis=1, keepdims=True)
    mag = (np.abs(q) @ np.abs(Kr).T) * scale
    D = ACC * np.where(causal, mag, 0.0).max(axis=1)
    dev = np.abs(Vr[None, :, :] - O_ref[:, None, :])
    mad = np.einsum("tj,tjd->td", wts, dev)
    absv = wts @ np.abs(Vr)
    # Terms whose P may be subnormal: more than 12 binades below the row maximum.
    sub = causal & ((logits - logits.max(axis=1, keepdims=True)) * math.log2(math.e) < -12.0)
    subdev = np.einsum("tj,tjd->td", sub.astype(np.float64), dev)
    fac = 2 * U8 / (1 - U8) + 2 * (np.exp(2 * D) - 1)
    tol = fac[:, None] * mad + 2.0 * 2.0 ** -16 * subdev + ACC * (absv + np.abs(O_ref)) + 2.0 ** -8 * np.abs(O_ref)
    return tol + 1e-5, D, sub.sum(axis=1)


def _check_attention(r, ref, w, rows):
    B = w.block_size
    scale = 1.0 / math.sqrt(w.head_dim)
    Qv, Kv, Vv = ref["q"][3], ref["k"][3], ref["v"][3]
    Og = H.bf16_tensor_to_f64(r["O"])
    lse = r["lse"].cpu().numpy()
    lists = H.gpu_rows(r["counts"], r["indices"], rows)
    worst_ratio, worst_err = 0.0, 0.0
    for (h, i), ids in lists.items():
        g = h // w.group
        O_ref = oracle.attention_rows(Qv[h], Kv[g], Vv[g], B, i, ids)
        s, e = i * B, min((i + 1) * B, w.seq_len)
        err = np.abs(Og[h, s:e] - O_ref)
        tol, D, n_sub = _bound(Qv[h], Kv[g], Vv[g], B, i, ids, O_ref, scale)
        worst_ratio = max(worst_ratio, float((err / tol).max()))
        worst_err = max(worst_err, float(err.max()))
        # LSE: natural log of the sum of exp(scaled logits) over the retained
        # causal keys; the GPU sums E4M3-rounded terms (relative error <= u)
        # of logits off by at most D.
        key_pos = np.concatenate([np.arange(b * B, min((b + 1) * B, w.seq_len)) for b in ids])
        lg = (Qv[h, s:e] @ Kv[g, key_pos].T) * scale
        lg = np.where(key_pos[None, :] <= np.arange(s, e)[:, None], lg, -np.inf)
        m = lg.max(axis=1)
        want = m + np.log(np.exp(lg - m[:, None]).sum(axis=1))
        lse_tol = np.log1p(U8 / (1 - U8) + 2.0 ** -16 * n_sub) + ACC + 2 * D + 1e-5
        bad = np.abs(lse[h, s:e] - want) - lse_tol
        assert (bad <= 0).all(), f"row {(h, i)} lse off by {bad.max():.3g} beyond its bound"
    return worst_err, worst_ratio


@pytest.mark.parametrize("variant", [
    dict(seq_len=1000, n_q_heads=4, n_kv_heads=2, seed=21, block_size=128),   # ragged tail, GQA 2:1
    dict(seq_len=2048, n_q_heads=2, n_kv_heads=1, seed=22, block_size=128),
    dict(seq_len=100, n_q_heads=2, n_kv_heads=2, seed=23, block_size=128),    # N < B
    dict(seq_len=1000, n_q_heads=4, n_kv_heads=2, seed=24, block_size=64),    # one 64-key PV step
    dict(seq_len=1500, n_q_heads=4, n_kv_heads=2, seed=25, block_size=256),   # two 128-key softmax steps
    dict(seq_len=200, n_q_heads=2, n_kv_heads=1, seed=26, block_size=256),    # N < B, one partial block
])
def test_fp8_pack_and_attention(variant):
    w = WORKLOADS["tiny-2k"].with_(name="fp8", needles_per_kv_head=2, **variant)
    _say(f"[fp8] B={w.block_size} N={w.seq_len} Hq={w.n_q_heads} Hkv={w.n_kv_heads}")
    r = _run(w)
    ref = _oracle_fp8(r["inp"])
    _check_pack(r, ref, w)
    rows = [(h, i) for h in range(w.n_q_heads) for i in range(w.n_blocks)]
    err, ratio = _check_attention(r, ref, w, rows)
    _say(f"[fp8] N={w.seq_len}: codes bit-exact; attention max-abs {err:.3e}, max err/bound {ratio:.3f}")
    assert ratio <= 1.0


@pytest.mark.parametrize("B", [64, 128, 256])
def test_fp8_full_selection_is_dense_attention_on_the_fp8_values(B):
    w = WORKLOADS["tiny-2k"].with_(name="fp8-dense", block_size=B, seq_len=1536, needles_per_kv_head=2, seed=24)
    r = _run(w, tau=(0.0, 0.0), forced=(1, 2, 0))
    counts = r["counts"].cpu().numpy()
    assert (counts == np.arange(w.n_blocks)[None, :] + 1).all()
    ref = _oracle_fp8(r["inp"])
    Og = H.bf16_tensor_to_f64(r["O"])
    for h in range(w.n_q_heads):
        dense = oracle.dense_causal_attention(ref["q"][3][h], ref["k"][3][h // w.group], ref["v"][3][h // w.group])
        assert np.abs(Og[h] - dense).max() <= 0.1
    err, ratio = _check_attention(r, ref, w, [(h, i) for h in range(w.n_q_heads) for i in range(w.n_blocks)])
    _say(f"[fp8] dense lists: max-abs {err:.3e}, max err/bound {ratio:.3f}")
    assert ratio <= 1.0


@pytest.mark.slow
def test_fp8_qwen3_32k_sampled():
    w = WORKLOADS["qwen3-30b-a3b-32k"]
    _say(f"[fp8] {w.name}")
    r = _run(w)
    ref = _oracle_fp8(r["inp"])
    f8 = r["f8"]
    amax = f8.amax.cpu().numpy().astype(np.float64)
    assert np.array_equal(amax, np.concatenate([ref["q"][0], ref["k"][0], ref["v"][0]]))
    assert np.array_equal(f8.Q8.cpu().numpy(), ref["q"][1]) and np.array_equal(f8.K8.cpu().numpy(), ref["k"][1])
    rows = H.sample_rows(w.n_q_heads, w.n_blocks, 10, seed=7, include=[(0, w.n_blocks - 1), (31, 100)])
    err, ratio = _check_attention(r, ref, w, rows)
    _say(f"[fp8] {w.name}: max-abs {err:.3e}, max err/bound {ratio:.3f}")
    assert ratio <= 1.0
