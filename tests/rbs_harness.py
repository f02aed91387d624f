"""Shared test plumbing: move seeded inputs to the GPU, run the HIP path through
the C ABI, and compare with the oracle under the parity rules.

Parity rules (tolerances are fixed here, in one place):
  centroids  per block |c_gpu - c|_2 / |c|_2 <= 1e-3 (|c| = 0: absolute 1e-5)
  radii      elementwise relative <= 1e-3
  beta       absolute <= 1e-3; quantiles relative <= 1e-3
  masks      identical, except non-forced blocks decided within 1e-3 of a
             threshold: with the oracle margin log S_b - log tau - max log S
             (natural log) of each branch, a block the oracle keeps may be
             dropped only if every branch that keeps it has margin <= 1e-3, and
             a block the oracle drops may be kept only if some branch has margin
             in [-1e-3, 0); those are counted and reported
  attention  max |O_gpu - O_oracle| <= 2e-2, with the oracle run in float64 on
             the GPU's own lists and the same bf16 inputs
"""

from __future__ import annotations

import math

import numpy as np

import oracle
from synth import f64_from_bf16_bits

CENTROID_RTOL = 1e-3
RADIUS_RTOL = 1e-3
BETA_ATOL = 1e-3
MARGIN_BAND = 1e-3
ATTN_ATOL = 2e-2


def to_device(bits: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def bf16_tensor_to_f64(t) -> np.ndarray:
    import torch
    return f64_from_bf16_bits(t.detach().view(torch.int16).cpu().numpy().view(np.uint16))


def run_stats(shape, K_dev):
    import paper_2609_20971_amd as rbs
    st = rbs.rbs_block_stats(shape, K_dev)
    return st


def check_stats(st, C, R, beta, rq):
    """Compare GPU statistics with the oracle's; return a small report."""
    Cg = st.centroids.cpu().numpy().astype(np.float64)
    Rg = st.radii.cpu().numpy().astype(np.float64)
    Bg = st.beta.cpu().numpy().astype(np.float64)
    Qg = st.quantiles.cpu().numpy().astype(np.float64)
    cn = np.linalg.norm(C, axis=-1)
    err = np.linalg.norm(Cg - C, axis=-1)
    rel = np.where(cn > 0, err / np.maximum(cn, 1e-300), err / 1e-5 * CENTROID_RTOL)
    assert rel.max() <= CENTROID_RTOL, f"centroid rel err {rel.max():.3g}"
    rrel = np.abs(Rg - R) / np.maximum(np.abs(R), 1e-30)
    rrel = np.where(R == 0, np.abs(Rg) / 1e-5 * RADIUS_RTOL, rrel)
    assert rrel.max() <= RADIUS_RTOL, f"radius rel err {rrel.max():.3g}"
    assert np.abs(Bg - beta).max() <= BETA_ATOL, f"beta abs err {np.abs(Bg - beta).max():.3g}"
    qrel = np.abs(Qg - rq) / np.maximum(np.abs(rq), 1e-30)
    qrel = np.where(rq == 0, np.abs(Qg) / 1e-5 * RADIUS_RTOL, qrel)
    assert qrel.max() <= RADIUS_RTOL, f"quantile rel err {qrel.max():.3g}"
    return {"centroid_rel": float(rel.max()), "radius_rel": float(rrel.max()),
            "beta_abs": float(np.abs(Bg - beta).max())}


def summary_parts(summary, n_kv_heads: int, n_blocks: int):
    """The written parts of a select-ready summary (f16 scaled centroids, fp32
    uplift, fp32 centroid norms; each part starts on a 256-byte boundary and
    the padding between them is never written), as byte views."""
    def up(x):
        return (x + 255) // 256 * 256
    n = n_kv_heads * n_blocks
    c_end = n * 128 * 2
    u_off = up(c_end)
    n_off = up(u_off + 4 * n)
    return summary[:c_end], summary[u_off:u_off + 4 * n], summary[n_off:n_off + 4 * n]


def summaries_equal(a, b, n_kv_heads: int, n_blocks: int) -> bool:
    import torch
    return all(torch.equal(x, y) for x, y in zip(summary_parts(a, n_kv_heads, n_blocks),
                                                 summary_parts(b, n_kv_heads, n_blocks)))


def gpu_rows(counts, indices, rows):
    """{(h, i): sorted list} from device counts/indices for the given rows."""
    cnt = counts.cpu().numpy()
    idx = indices.cpu().numpy()
    out = {}
    for (h, i) in rows:
        base = i * (i + 1) // 2
        out[(h, i)] = idx[h, base:base + cnt[h, i]].tolist()
    return out


def check_lists(lists, n_blocks, n_sink, n_local, n_recent):
    """Structural invariants of every list: ascending, unique, causal, forced."""
    for (h, i), ids in lists.items():
        assert ids == sorted(set(ids)), f"row {(h, i)} not ascending/unique"
        assert all(0 <= b <= i for b in ids), f"row {(h, i)} has non-causal ids"
        forced = np.nonzero(oracle.forced_blocks(i, n_blocks, n_sink, n_local, n_recent))[0]
        assert set(forced.tolist()) <= set(ids), f"row {(h, i)} misses forced blocks"


def compare_masks(gpu_lists, oracle_rows):
    """Return (n_rows, n_blocks_compared, near_flips); assert no other flip."""
    near = 0
    compared = 0
    for key, ids in gpu_lists.items():
        ref = oracle_rows[key]
        g = np.zeros(ref["final"].shape[0], dtype=bool)
        g[ids] = True
        compared += g.shape[0]
        diff = np.nonzero(g != ref["final"])[0]
        for b in diff:
            assert not ref["forced"][b], f"forced block {b} differs in row {key}"
            if "margin" in ref:  # single-branch supporting selector
                margins = [ref["margin"][b]]
            else:
                margins = [ref["margin_base"][b], ref["margin_rescue"][b]]
            if ref["final"][b]:
                # The oracle keeps it, the GPU drops it: every branch that keeps
                # it must do so from inside the band.
                ok = all(m <= MARGIN_BAND for m in margins if m >= 0)
            else:
                # The GPU keeps it, the oracle drops it: some branch must miss
                # its threshold by no more than the band.
                ok = any(-MARGIN_BAND <= m < 0 for m in margins)
            assert ok, (f"row {key} block {b}: gpu={bool(g[b])} oracle={bool(ref['final'][b])} "
                        f"margins {', '.join(f'{m:.3g}' for m in margins)}")
            near += 1
    return len(gpu_lists), compared, near


def attention_reference(Qh, Kg, Vg, block_size, row_lists, scale=None):
    return oracle.attention_on_mask(Qh, Kg, Vg, block_size, row_lists, scale)


def max_abs_attention_error(O_gpu_f64, Qf, Kf, Vf, group, block_size, lists, n_tokens):
    """Max |O_gpu - O_oracle| over the given rows (oracle on the GPU's lists)."""
    worst = 0.0
    by_head = {}
    for (h, i), ids in lists.items():
        by_head.setdefault(h, {})[i] = ids
    for h, rows in by_head.items():
        g = h // group
        ref = oracle.attention_on_mask(Qf[h], Kf[g], Vf[g], block_size, rows)
        for i, o in ref.items():
            s, e = i * block_size, min((i + 1) * block_size, n_tokens)
            worst = max(worst, float(np.abs(O_gpu_f64[h, s:e] - o).max()))
    return worst


def sample_rows(n_heads, n_blocks, k, seed=0, include=()):
    rng = np.random.default_rng(seed)
    rows = set(include)
    rows |= {(int(rng.integers(n_heads)), int(rng.integers(n_blocks))) for _ in range(k)}
    rows.add((0, 0))
    rows.add((n_heads - 1, n_blocks - 1))
    return sorted(rows)


def scale_default(d):
    return 1.0 / math.sqrt(d)
