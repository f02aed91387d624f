"""Float64 oracle of the RBS-Attention sparse-prefill path (test infrastructure only).

Written from the paper's definitions, step by step, with no blocking or fusion
beyond what the definitions state.  Conventions (readings of points the paper
leaves open are marked READING and listed in the design notes):

* Q is [H_q][N][d], K and V are [H_kv][N][d]; query head h uses KV head
  h // (H_q // H_kv) (READING: selection is made per query head).
* Blocks: token range [b B, min((b+1) B, N)); the same partition for queries
  and keys (Sec. 2.1, Sec. 4.4: query and key block size are equal).
* Candidates of query block i are key blocks 0..i (READING: the diagonal block
  and forced blocks take part in the maximum of the relative threshold).
"""

from __future__ import annotations

import math

import numpy as np


# ---------------------------------------------------------------- partition

def block_ranges(n_tokens: int, block_size: int) -> list:
    """[(start, end)] of the M = ceil(N / B) blocks (Sec. 2.1)."""
    return [(s, min(s + block_size, n_tokens)) for s in range(0, n_tokens, block_size)]


# ---------------------------------------------------------------- Sec. 3.1

def block_stats(K: np.ndarray, block_size: int):
    """Centroid c_b = mean of the block's keys and radius r_b = max_k |k - c_b|_2.

    Sec. 3.1, centroid and maximum-radius equations; Algorithm 1, first loop.
    K: [H_kv][N][d] float64.  Returns centroids [H_kv][M][d], radii [H_kv][M].
    The mean divides by the block's actual key count |K_b| (a short last block
    uses its own count).
    """
    K = np.asarray(K, dtype=np.float64)
    H, N, d = K.shape
    ranges = block_ranges(N, block_size)
    C = np.zeros((H, len(ranges), d))
    R = np.zeros((H, len(ranges)))
    for g in range(H):
        for b, (s, e) in enumerate(ranges):
            keys = K[g, s:e]
            c = keys.sum(axis=0) / (e - s)
            C[g, b] = c
            R[g, b] = np.sqrt(((keys - c) ** 2).sum(axis=1)).max()
    return C, R


def quantile_type7(values, p: float) -> float:
    """Sample quantile by linear interpolation between order statistics.

    READING: the paper writes quantile(r, p) without naming an estimator; this
    is the common "type 7" rule: with x sorted ascending (0-based) and
    h = (n - 1) p, Q = x[floor h] + (h - floor h) (x[floor h + 1] - x[floor h]).
    """
    x = sorted(float(v) for v in values)
    n = len(x)
    h = (n - 1) * p
    lo = int(math.floor(h))
    hi = min(lo + 1, n - 1)
    return x[lo] + (h - lo) * (x[hi] - x[lo])


def radius_quantiles(R: np.ndarray):
    """Per KV head: r_low = quantile(r, 0.5), r_high = quantile(r, 0.9) over
    all M block radii of the prompt (Sec. 3.1; Algorithm 1).  Returns [H_kv][2]."""
    R = np.asarray(R, dtype=np.float64)
    return np.array([[quantile_type7(R[g], 0.5), quantile_type7(R[g], 0.9)]
                     for g in range(R.shape[0])])


def rescue_coefficients(R: np.ndarray):
    """beta_b = clamp((r_b - r_low) / (r_high - r_low), 0, 1) (Sec. 3.1, Eq. beta).

    READING for r_high <= r_low, where the paper leaves beta undefined: the
    limit of the clamp, beta_b = 1 if r_b > r_low else 0.
    Returns (beta [H_kv][M], quantiles [H_kv][2]).
    """
    R = np.asarray(R, dtype=np.float64)
    rq = radius_quantiles(R)
    beta = np.zeros_like(R)
    for g in range(R.shape[0]):
        r_low, r_high = rq[g]
        if r_high > r_low:
            beta[g] = np.clip((R[g] - r_low) / (r_high - r_low), 0.0, 1.0)
        else:
            beta[g] = (R[g] > r_low).astype(np.float64)
    return beta, rq


# ---------------------------------------------------------------- Sec. 3.2

def branch_logits(Qi: np.ndarray, C: np.ndarray, R: np.ndarray, beta: np.ndarray,
                  n_candidates: int):
    """Token-level logits of both branches against candidates 0..n-1.

    Qi: [n_i][d] queries of one query block; C, R, beta: one KV head's
    statistics.  Base logit l_base(q, b) = q . c_b (Sec. 3.2, Eq. base_score);
    rescue logit l_rescue(q, b) = q . c_b + |q|_2 r_b beta_b (Eq. rescue_score).
    Returns (l_base, l_rescue), each [n_i][n_candidates], unscaled.
    """
    Qi = np.asarray(Qi, dtype=np.float64)
    cand = C[:n_candidates]
    l_base = Qi @ cand.T
    qnorm = np.sqrt((Qi * Qi).sum(axis=1))
    l_rescue = l_base + qnorm[:, None] * (R[:n_candidates] * beta[:n_candidates])[None, :]
    return l_base, l_rescue


def branch_log_scores(Qi: np.ndarray, C: np.ndarray, R: np.ndarray, beta: np.ndarray,
                      n_candidates: int):
    """Query-block aggregated scores of both branches for candidates 0..n-1.

    The logits of branch_logits are scaled by 1/sqrt(d) and aggregated over the
    block's tokens with the shared shift of Sec. 3.2, Eq. block_aggregation:
        m = max_b max_t l(q_t, b)/sqrt(d),  S_b = sum_t exp(l(q_t, b)/sqrt(d) - m).
    Returns (log S_base, log S_rescue) over the candidates, with log 0 = -inf.
    """
    d = np.asarray(Qi).shape[1]
    out = []
    for logits in branch_logits(Qi, C, R, beta, n_candidates):
        x = logits / math.sqrt(d)
        m = x.max()
        S = np.exp(x - m).sum(axis=0)
        with np.errstate(divide="ignore"):
            out.append(np.log(S))
    return out[0], out[1]


def forced_blocks(i: int, n_blocks: int, n_sink: int, n_local: int, n_recent: int) -> np.ndarray:
    """Forced set for query block i over candidates 0..i (Sec. 3.2, union).

    READINGS: sink = the first n_sink key blocks; local window = the n_local
    blocks ending at the diagonal; recent = the last n_recent query blocks keep
    every causal candidate.
    """
    f = np.zeros(i + 1, dtype=bool)
    f[:min(n_sink, i + 1)] = True
    f[max(0, i - n_local + 1):i + 1] = True
    if i >= n_blocks - n_recent:
        f[:] = True
    return f


def _threshold(log_s: np.ndarray, alpha: float):
    """Eq. branch_thresholds in log space: S_b >= alpha max S  <=>
    log S_b >= log alpha + max log S.  Returns (mask, margin) where margin is
    log S_b - log alpha - max log S (the mask is margin >= 0)."""
    top = log_s.max()
    if alpha <= 0.0:
        return np.ones(log_s.shape, dtype=bool), np.full(log_s.shape, np.inf)
    with np.errstate(invalid="ignore"):
        margin = log_s - math.log(alpha) - top
    margin = np.where(np.isnan(margin), -np.inf, margin)
    return margin >= 0.0, margin


def select_row(Qi, C, R, beta, i: int, n_blocks: int, tau_base: float, tau_rescue: float,
               n_sink: int, n_local: int, n_recent: int) -> dict:
    """Final mask of query block i: M_base U M_rescue U forced (Sec. 3.2)."""
    log_b, log_r = branch_log_scores(Qi, C, R, beta, i + 1)
    m_base, margin_base = _threshold(log_b, tau_base)
    m_res, margin_res = _threshold(log_r, tau_rescue)
    forced = forced_blocks(i, n_blocks, n_sink, n_local, n_recent)
    return {
        "base": m_base,
        "rescue": m_res,
        "forced": forced,
        "final": m_base | m_res | forced,
        "log_s_base": log_b,
        "log_s_rescue": log_r,
        "margin_base": margin_base,
        "margin_rescue": margin_res,
    }


def select(Q, C, R, beta, block_size: int, tau_base: float, tau_rescue: float,
           n_sink: int, n_local: int, n_recent: int, rows=None) -> dict:
    """Run select_row for every (query head, query block) in `rows` (default:
    all).  Q: [H_q][N][d] real values; C, R, beta: per KV head.
    Returns {(h, i): row dict}."""
    H_q, n_tokens = Q.shape[0], Q.shape[1]
    group = H_q // C.shape[0]
    ranges = block_ranges(n_tokens, block_size)
    M = len(ranges)
    if rows is None:
        rows = [(h, i) for h in range(H_q) for i in range(M)]
    out = {}
    for (h, i) in rows:
        g = h // group
        s, e = ranges[i]
        out[(h, i)] = select_row(np.asarray(Q[h, s:e], dtype=np.float64), C[g], R[g], beta[g],
                                 i, M, tau_base, tau_rescue, n_sink, n_local, n_recent)
    return out


# ------------------------------------- supporting selectors (Table selector_ablation)
#
# The paper compares the dual-branch selector with three alternatives in the
# same prefill backend (Sec. 4, supporting selector comparison; App.
# geometry): centroid-only scoring, the unattenuated full-L2 bound, and a
# Quest-style coordinate-wise box.  READINGS: each alternative is a single
# branch whose token-level logits are aggregated over the query block exactly
# as in Eq. block_aggregation; centroid-only and full-L2 keep the relative
# threshold of Eq. branch_thresholds, the Quest-style policy keeps a fixed
# budget (the k = max(1, ceil(rho |C_i|)) highest scores, ties with the k-th
# kept); forced blocks are added to every variant.

SELECTOR_VARIANTS = ("centroid", "full_l2", "box")


def block_box(K: np.ndarray, block_size: int):
    """Coordinate-wise key minima a_b and maxima u_b of every block (App.
    geometry, Eq. quest_box), returned as the box centre v_b = (u_b + a_b)/2
    and half-width h_b = (u_b - a_b)/2, each [H_kv][M][d]."""
    K = np.asarray(K, dtype=np.float64)
    H, N, d = K.shape
    ranges = block_ranges(N, block_size)
    Vc = np.zeros((H, len(ranges), d))
    Hw = np.zeros((H, len(ranges), d))
    for g in range(H):
        for b, (s, e) in enumerate(ranges):
            lo = K[g, s:e].min(axis=0)
            hi = K[g, s:e].max(axis=0)
            Vc[g, b] = (hi + lo) / 2.0
            Hw[g, b] = (hi - lo) / 2.0
    return Vc, Hw


def variant_logits(Qi: np.ndarray, C: np.ndarray, R: np.ndarray, Vc: np.ndarray, Hw: np.ndarray,
                   n_candidates: int, variant: str) -> np.ndarray:
    """Token-level logits [n_i][n_candidates] (unscaled) of one supporting selector:
        centroid  q . c_b                                  (Eq. base_score)
        full_l2   q . c_b + |q|_2 r_b                      (Eq. full_l2_bound)
        box       sum_j max(q_j a_bj, q_j u_bj)            (Eq. quest_box)
    One KV head's statistics; Vc, Hw (box centre and half-width) are used by
    the box only and may be None otherwise."""
    Qi = np.asarray(Qi, dtype=np.float64)
    n = n_candidates
    if variant == "centroid":
        return Qi @ C[:n].T
    if variant == "full_l2":
        qnorm = np.sqrt((Qi * Qi).sum(axis=1))
        return Qi @ C[:n].T + qnorm[:, None] * R[:n][None, :]
    if variant == "box":
        lo = Vc[:n] - Hw[:n]
        hi = Vc[:n] + Hw[:n]
        return np.maximum(Qi[:, None, :] * lo[None, :, :], Qi[:, None, :] * hi[None, :, :]).sum(axis=2)
    raise ValueError(variant)


def variant_log_scores(Qi, C, R, Vc, Hw, n_candidates: int, variant: str) -> np.ndarray:
    """log S_b of a supporting selector: the logits of variant_logits scaled by
    1/sqrt(d) and aggregated over the block's tokens with the shared shift of
    Eq. block_aggregation (log 0 = -inf)."""
    d = np.asarray(Qi).shape[1]
    x = variant_logits(Qi, C, R, Vc, Hw, n_candidates, variant) / math.sqrt(d)
    m = x.max()
    S = np.exp(x - m).sum(axis=0)
    with np.errstate(divide="ignore"):
        return np.log(S)


def top_fraction(log_s: np.ndarray, rho: float):
    """Fixed-budget selection: the k = max(1, ceil(rho n)) largest scores, ties
    with the k-th kept.  Returns (mask, margin) with margin = log S_b minus the
    k-th largest log S (the mask is margin >= 0)."""
    n = log_s.shape[0]
    k = min(n, max(1, int(math.ceil(rho * n - 1e-12))))
    kth = np.sort(log_s)[::-1][k - 1]
    with np.errstate(invalid="ignore"):
        margin = log_s - kth
    margin = np.where(np.isnan(margin), -np.inf, margin)
    return margin >= 0.0, margin


def select_variant_row(Qi, C, R, Vc, Hw, i: int, n_blocks: int, variant: str, param: float,
                       n_sink: int, n_local: int, n_recent: int) -> dict:
    """Mask of query block i under a supporting selector: its single branch
    (relative threshold param for centroid / full_l2, budget fraction param for
    box) united with the forced blocks."""
    log_s = variant_log_scores(Qi, C, R, Vc, Hw, i + 1, variant)
    if variant == "box":
        mask, margin = top_fraction(log_s, param)
    else:
        mask, margin = _threshold(log_s, param)
    forced = forced_blocks(i, n_blocks, n_sink, n_local, n_recent)
    return {"branch": mask, "forced": forced, "final": mask | forced, "log_s": log_s, "margin": margin}


def select_variant(Q, C, R, Vc, Hw, block_size: int, variant: str, param: float,
                   n_sink: int, n_local: int, n_recent: int, rows=None) -> dict:
    """select_variant_row for every (query head, query block) in `rows`."""
    H_q, n_tokens = Q.shape[0], Q.shape[1]
    group = H_q // C.shape[0]
    ranges = block_ranges(n_tokens, block_size)
    M = len(ranges)
    if rows is None:
        rows = [(h, i) for h in range(H_q) for i in range(M)]
    out = {}
    for (h, i) in rows:
        g = h // group
        s, e = ranges[i]
        out[(h, i)] = select_variant_row(np.asarray(Q[h, s:e], dtype=np.float64), C[g], R[g],
                                         None if Vc is None else Vc[g], None if Hw is None else Hw[g],
                                         i, M, variant, param, n_sink, n_local, n_recent)
    return out


# ---------------------------------------------------------------- Sec. 3.3

def attention_rows(Qh, Kg, Vg, block_size: int, i: int, kv_blocks, scale: float | None = None):
    """Attention of query block i over the keys of the retained blocks, with
    token-level causal masking and softmax over the retained causal keys
    (Sec. 3.3; Eq. (1) restricted to the retained keys).  Float64.
    Returns [n_i][d]; a query with no retained causal key gets zeros."""
    Qh = np.asarray(Qh, dtype=np.float64)
    N, d = Kg.shape
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(d)
    s, e = i * block_size, min((i + 1) * block_size, N)
    key_pos = np.concatenate([np.arange(b * block_size, min((b + 1) * block_size, N))
                              for b in sorted(kv_blocks)]) if len(kv_blocks) else np.zeros(0, int)
    keys = np.asarray(Kg[key_pos], dtype=np.float64)
    vals = np.asarray(Vg[key_pos], dtype=np.float64)
    out = np.zeros((e - s, d))
    for t in range(s, e):
        keep = key_pos <= t
        if not keep.any():
            continue
        logits = keys[keep] @ Qh[t] * scale
        p = np.exp(logits - logits.max())
        out[t - s] = (p @ vals[keep]) / p.sum()
    return out


def attention_on_mask(Qh, Kg, Vg, block_size: int, row_blocks: dict, scale: float | None = None):
    """Sparse attention for one query head over {i: retained key blocks}.
    Returns {i: [n_i][d]}."""
    return {i: attention_rows(Qh, Kg, Vg, block_size, i, blocks, scale)
            for i, blocks in row_blocks.items()}


def dense_causal_attention(Qh, Kg, Vg, scale: float | None = None):
    """Brute-force causal softmax attention, Eq. (1): for every token t,
    O_t = sum_{j<=t} softmax_j(q_t . k_j * scale) v_j.  Float64, O(N^2 d)."""
    Qh = np.asarray(Qh, dtype=np.float64)
    Kg = np.asarray(Kg, dtype=np.float64)
    Vg = np.asarray(Vg, dtype=np.float64)
    N, d = Qh.shape
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((N, d))
    for t in range(N):
        logits = Kg[:t + 1] @ Qh[t] * scale
        w = np.exp(logits - logits.max())
        out[t] = (w / w.sum()) @ Vg[:t + 1]
    return out


# ---------------------------------------------------------------- Sec. 4.4

def density(final_masks) -> float:
    """Actual density: selected valid causal block pairs / all valid causal block
    pairs, forced blocks and branch overlap counted once (Sec. 4.4).
    final_masks: iterable of per-(head, query block) boolean rows over 0..i."""
    selected = 0
    total = 0
    for row in final_masks:
        row = np.asarray(row, dtype=bool)
        selected += int(row.sum())
        total += row.shape[0]
    return selected / total if total else 0.0


# ---------------------------------------------------------------- list <-> mask

def lists_from_masks(masks: dict, n_heads: int, n_blocks: int):
    """Ascending per-row index lists in the triangular packing: row (h, i)
    starts at i (i + 1) / 2 and holds counts[h][i] block ids."""
    cap = n_blocks * (n_blocks + 1) // 2
    counts = np.zeros((n_heads, n_blocks), dtype=np.int32)
    indices = np.full((n_heads, cap), -1, dtype=np.int32)
    for (h, i), row in masks.items():
        ids = np.nonzero(np.asarray(row, dtype=bool))[0]
        counts[h, i] = len(ids)
        base = i * (i + 1) // 2
        indices[h, base:base + len(ids)] = ids
    return counts, indices


def masks_from_lists(counts, indices, rows):
    """Inverse of lists_from_masks for the given (h, i) rows."""
    out = {}
    for (h, i) in rows:
        base = i * (i + 1) // 2
        row = np.zeros(i + 1, dtype=bool)
        row[np.asarray(indices[h, base:base + counts[h, i]], dtype=np.int64)] = True
        out[(h, i)] = row
    return out


# ---------------------------------------------------------------- batches
#
# App. "Additional A100 System Measurements", prompt throughput: a batch of
# prompts is a set of independent causal sequences; none is concatenated into
# another.  Every per-prompt quantity -- the block partition, the radius
# quantiles and beta (the prompt's own radius distribution, Sec. 3.1), the
# candidates, the causal attention -- is that of the sequence alone.  Layout of
# a batch: the sequences packed along the token axis, and the block arrays
# holding the sequences' blocks one after another.

def batch_offsets(seq_tokens) -> list:
    """Token offsets of the sequences: 0, n_0, n_0 + n_1, ..., T."""
    out = [0]
    for n in seq_tokens:
        out.append(out[-1] + int(n))
    return out


def batch_sequences(X, seq_tokens) -> list:
    """[X[:, t_s : t_s + n_s]] for every sequence s of a packed [H][T][d] batch."""
    off = batch_offsets(seq_tokens)
    assert off[-1] == X.shape[1], "sequence lengths must add up to the packed length"
    return [X[:, off[s]:off[s + 1]] for s in range(len(seq_tokens))]


def batch_block_stats(K, seq_tokens, block_size: int):
    """block_stats and rescue_coefficients of every sequence alone, laid out
    as the batch's block arrays: C [H_kv][M_tot][d], R and beta [H_kv][M_tot],
    quantiles [n_seqs][H_kv][2]."""
    parts = [block_stats(Ks, block_size) for Ks in batch_sequences(K, seq_tokens)]
    coeffs = [rescue_coefficients(R) for (_, R) in parts]
    C = np.concatenate([c for (c, _) in parts], axis=1)
    R = np.concatenate([r for (_, r) in parts], axis=1)
    beta = np.concatenate([b for (b, _) in coeffs], axis=1)
    rq = np.stack([q for (_, q) in coeffs])
    return C, R, beta, rq


def batch_select(Q, K, seq_tokens, block_size: int, tau_base: float, tau_rescue: float,
                 n_sink: int, n_local: int, n_recent: int, rows=None) -> dict:
    """select on every sequence alone.  rows: {s: [(h, i)]} (default: every
    row of every sequence).  Returns {s: {(h, i): row dict}}, i local to s."""
    Qs, Ks = batch_sequences(Q, seq_tokens), batch_sequences(K, seq_tokens)
    out = {}
    for s in range(len(seq_tokens)):
        if rows is not None and s not in rows:
            continue
        C, R = block_stats(Ks[s], block_size)
        beta, _ = rescue_coefficients(R)
        out[s] = select(Qs[s], C, R, beta, block_size, tau_base, tau_rescue, n_sink, n_local, n_recent,
                        rows=None if rows is None else rows[s])
    return out


def batch_attention_on_mask(Q, K, V, seq_tokens, block_size: int, row_blocks: dict,
                            scale: float | None = None) -> dict:
    """attention_on_mask on every sequence alone.  row_blocks: {s: {h: {i:
    retained blocks}}}, i and the blocks local to s.  Returns {s: {h: {i: O}}}."""
    Qs, Ks, Vs = (batch_sequences(X, seq_tokens) for X in (Q, K, V))
    group = Q.shape[0] // K.shape[0]
    return {s: {h: attention_on_mask(Qs[s][h], Ks[s][h // group], Vs[s][h // group], block_size, rows, scale)
                for h, rows in heads.items()}
            for s, heads in row_blocks.items()}


# ---------------------------------------------------------------- FP8 inputs
#
# Attention on FP8 inputs (the paper's models are FP8 checkpoints, Sec. 4.1;
# the precision of their attention is not stated).  The format is E4M3 as
# the OCP 8-bit floating-point specification defines it: 1 sign bit, 4
# exponent bits with bias 7, 3 mantissa bits; subnormals (m / 8) 2^-6; the
# largest finite magnitude 448 (S.1111.110); no infinities.  READINGS: each
# head is scaled so that its largest |x| maps to 448 (inv = 448 / amax and
# dequantisation amax / 448, both rounded to float32, x * inv rounded to
# float32 before the conversion), conversion rounds to nearest with ties to
# even and saturates at 448.  Attention on FP8 inputs is attention_on_mask on
# the dequantised values.

E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """Value of each E4M3 code (uint8 array), float64; the two NaN codes decode to nan."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * 2.0 ** (e - 7))
    mag = np.where((c & 0x7f) == 0x7f, np.nan, mag)
    return sign * mag


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code of each finite value (ties to even mantissa),
    magnitudes above 448 saturating to 448.  Returns uint8."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    out = np.zeros(a.shape, dtype=np.int64)
    sub = a < 2.0 ** -6
    # Subnormal range: a multiple of 2^-9, rounded half to even (np.rint).
    out[sub] = np.rint(a[sub] * 2.0 ** 9).astype(np.int64)
    nrm = ~sub
    if nrm.any():
        an = a[nrm]
        e = np.floor(np.log2(an)).astype(np.int64)
        # Guard the floor of log2 at exact powers of two.
        e = np.where(2.0 ** e > an, e - 1, e)
        e = np.where(2.0 ** (e + 1) <= an, e + 1, e)
        q = np.rint((an / 2.0 ** e - 1.0) * 8.0).astype(np.int64)  # mantissa in eighths, half to even
        carry = q == 8
        e = np.where(carry, e + 1, e)
        q = np.where(carry, 0, q)
        out[nrm] = ((e + 7) << 3) | q
    out = np.where(np.signbit(x), out | 0x80, out)
    return out.astype(np.uint8)


def fp8_amax(X) -> np.ndarray:
    """Largest |x| of every head of X [H][N][d]."""
    X = np.asarray(X, dtype=np.float64)
    return np.abs(X).reshape(X.shape[0], -1).max(axis=1)


def fp8_quantize(X, amax):
    """E4M3 codes of X [H][N][d] with the per-head scaling above, and the
    float32 dequantisation scale of every head.  Returns (codes uint8, deq)."""
    X = np.asarray(X, dtype=np.float64)
    codes = np.empty(X.shape, dtype=np.uint8)
    deq = np.empty(X.shape[0], dtype=np.float64)
    for h in range(X.shape[0]):
        am = np.float32(amax[h])
        inv = np.float32(448.0) / am if am > 0 else np.float32(1.0)
        deq[h] = float(am / np.float32(448.0)) if am > 0 else 1.0
        y = (X[h].astype(np.float32) * inv).astype(np.float32)
        codes[h] = e4m3_encode(y)
    return codes, deq


def fp8_dequantize(codes, deq) -> np.ndarray:
    """Values of E4M3 codes [H][N][d] times each head's scale, float64."""
    return e4m3_decode(codes) * np.asarray(deq, dtype=np.float64)[:, None, None]
