"""The attention's first pass fixes the softmax reference from the first listed
block and handles later, larger logits in three ways: exponentials above 1
within its range, exact power-of-two rescales of O and the denominator, and,
past its range, a restart of the item with the running maximum that the
workgroup decides at the end of the offending block.  Each case below puts
key blocks at chosen logits (log2 units, Sec. 3.3's scaled dot product times
log2 e) so that one of these takes place, then checks O and LSE against the
float64 definition, Eq. (1), on dense lists and on short explicit lists."""

from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
from synth import bf16_bits_from_f32, f64_from_bf16_bits
from tests import rbs_harness as H

pytestmark = pytest.mark.gpu

N, B, D, HQ, HKV = 1024, 64, 128, 2, 1
M = N // B
SCALE_LOG2 = math.log2(math.e) / math.sqrt(D)

# Logit of each key block (log2 units) for queries along u; unlisted blocks sit near 0.
CASES = {
    # +20 per block: the denominator passes 2^32 every few blocks (power-of-two rescales).
    "climb": {b: 20.0 * b for b in range(M)},
    # Block 5 far above block 0, inside the reference's margin: no restart.
    "jump_within": {5: 90.0},
    # Block 5 beyond any fp32 exponential from block 0's reference: restart at block 5.
    "jump_beyond": {5: 200.0},
    # The same jump in the last block of every row that reaches it: the pass ends there.
    "jump_last": {M - 1: 200.0},
}


def _inputs(case: str):
    rng = np.random.default_rng(77)
    u = rng.standard_normal(D)
    u /= np.linalg.norm(u)
    q = np.broadcast_to(u, (HQ, N, D)) + 0.01 * rng.standard_normal((HQ, N, D))
    k = 0.05 * rng.standard_normal((HKV, N, D))
    for b, logit in CASES[case].items():
        k[:, b * B:(b + 1) * B] += u * (logit / SCALE_LOG2)
    v = rng.standard_normal((HKV, N, D))
    to_bits = lambda x: bf16_bits_from_f32(np.ascontiguousarray(x, dtype=np.float32))
    return {"q": to_bits(q), "k": to_bits(k), "v": to_bits(v)}


# P is rounded to bf16 (unit roundoff 2^-8) before the denominator sums it, so
# the LSE may differ from the definition by up to log(1 + 2^-8); fp32 adds a
# relative 1e-6 at these magnitudes (up to ~210 in natural-log units).
LSE_TOL = math.log1p(2.0 ** -8)


def _lse_ok(got, ref):
    return abs(got - ref) <= LSE_TOL + 1e-6 * abs(ref)


def _lse_ref(Qh, Kg, t, key_pos):
    x = Kg[key_pos[key_pos <= t]] @ Qh[t] / math.sqrt(D)
    return x.max() + math.log(np.exp(x - x.max()).sum())


def _lists(rows: dict):
    """counts [HQ][M] and triangular indices [HQ][M(M+1)/2] for {i: blocks}, the same for both heads."""
    counts = np.zeros((HQ, M), dtype=np.int32)
    indices = np.zeros((HQ, M * (M + 1) // 2), dtype=np.int32)
    for i, blocks in rows.items():
        base = i * (i + 1) // 2
        counts[:, i] = len(blocks)
        indices[:, base:base + len(blocks)] = sorted(blocks)
    return counts, indices


@pytest.mark.parametrize("case", list(CASES))
def test_fixed_reference_cases_match_the_definition(case):
    import torch
    import paper_2609_20971_amd as rbs
    print(f"[softmax-ref] {case}", flush=True)
    inp = _inputs(case)
    shape = rbs.make_shape(N, HQ, HKV, B)
    Qd, Kd, Vd = (H.to_device(inp[x]) for x in ("q", "k", "v"))
    Qf, Kf, Vf = (f64_from_bf16_bits(inp[x]) for x in ("q", "k", "v"))

    # Dense lists: every causal block, ascending.
    counts, indices = rbs.rbs_dense_indices(shape)
    lse = torch.empty((HQ, N), dtype=torch.float32, device="cuda")
    O = rbs.rbs_sparse_prefill(shape, Qd, Kd, Vd, counts, indices, 0.0, lse=lse)
    torch.cuda.synchronize()
    Og, lg = H.bf16_tensor_to_f64(O), lse.cpu().numpy()
    all_keys = np.arange(N)
    for h in range(HQ):
        ref = oracle.dense_causal_attention(Qf[h], Kf[0], Vf[0])
        assert np.abs(Og[h] - ref).max() <= H.ATTN_ATOL, (case, h)
        for t in range(0, N, 37):
            assert _lse_ok(lg[h, t], _lse_ref(Qf[h], Kf[0], t, all_keys)), (case, h, t)

    # Short lists: the sink, one middle block and the diagonal.
    rows = {i: sorted({0, min(5, i), i}) for i in range(M)}
    c_np, i_np = _lists(rows)
    counts = torch.from_numpy(c_np).cuda()
    indices = torch.from_numpy(i_np).cuda()
    O = rbs.rbs_sparse_prefill(shape, Qd, Kd, Vd, counts, indices, 0.0, lse=lse)
    torch.cuda.synchronize()
    Og, lg = H.bf16_tensor_to_f64(O), lse.cpu().numpy()
    for h in range(HQ):
        for i, blocks in rows.items():
            ref = oracle.attention_rows(Qf[h], Kf[0], Vf[0], B, i, blocks)
            assert np.abs(Og[h, i * B:(i + 1) * B] - ref).max() <= H.ATTN_ATOL, (case, h, i)
            key_pos = np.concatenate([np.arange(b * B, (b + 1) * B) for b in blocks])
            for t in range(i * B, (i + 1) * B, 29):
                assert _lse_ok(lg[h, t], _lse_ref(Qf[h], Kf[0], t, key_pos)), (case, h, i, t)
