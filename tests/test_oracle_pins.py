"""Pins of the float64 oracle against what the paper and mathematics fix.

Each test names the passage it follows.  None of them compares the oracle with
itself: expected values are hand-worked closed forms (tests/golden), library
routines for special cases, inequalities, invariances or brute force.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from tests.conftest import GOLDEN


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _case_rows(case, tau_base=None, tau_rescue=None):
    K = np.array(case["keys"], dtype=np.float64)[None]
    Q = np.array(case["queries"], dtype=np.float64)[None]
    B = case["block_size"]
    C, R = oracle.block_stats(K, B)
    beta, rq = oracle.rescue_coefficients(R)
    rows = oracle.select(Q, C, R, beta, B,
                         case.get("tau_base", 0.5) if tau_base is None else tau_base,
                         case.get("tau_rescue", 0.5) if tau_rescue is None else tau_rescue,
                         case["n_sink"], case["n_local"], case["n_recent"])
    return C, R, beta, rq, rows


def _ids(mask):
    return [int(x) for x in np.nonzero(mask)[0]]


# ------------------------------------------------------------ hand-worked cases

def test_needle_case():
    """Sec. 2.3 / 3.1 / 3.2: a needle diluted by noise is lost by the centroid
    score and recovered by the radius uplift."""
    case = _load("needle_case.json")
    ex = case["expected"]
    C, R, beta, rq, rows = _case_rows(case)
    np.testing.assert_allclose(C[0], ex["centroids"], atol=1e-15)
    np.testing.assert_allclose(R[0], ex["radii"], atol=1e-15)
    np.testing.assert_allclose(rq[0], [ex["r_low"], ex["r_high"]], rtol=1e-14)
    np.testing.assert_allclose(beta[0], ex["beta"], atol=1e-15)
    r2 = rows[(0, 2)]
    np.testing.assert_allclose(np.exp(r2["log_s_base"] - r2["log_s_base"].max()), ex["row2_base_ratio"], rtol=1e-12)
    np.testing.assert_allclose(np.exp(r2["log_s_rescue"] - r2["log_s_rescue"].max()), ex["row2_rescue_ratio"], rtol=1e-12)
    assert _ids(r2["base"]) == ex["row2_base"]
    assert _ids(r2["rescue"]) == ex["row2_rescue"]
    assert [_ids(rows[(0, i)]["final"]) for i in range(3)] == ex["final_rows"]
    assert _ids(r2["base"] | r2["forced"]) == ex["centroid_only_row2"]
    # The needle's logit meets the full L2 bound exactly (App. E).
    q = np.array(case["queries"][8], dtype=np.float64)
    needle = np.array(case["keys"][0], dtype=np.float64)
    assert q @ needle == ex["needle_logit"]
    assert q @ C[0, 0] + np.linalg.norm(q) * R[0, 0] == ex["needle_l2_bound"]


def test_aggregation_sums_exponentials_over_tokens():
    """Sec. 3.2 Eq. block_aggregation: the block score sums exp(logit/sqrt d)
    over the block's tokens (not a max, not a mean logit)."""
    case = _load("aggregation_case.json")
    ex = case["expected"]
    C, R, beta, rq, rows = _case_rows(case, 0.15, 0.15)
    np.testing.assert_allclose(beta[0], ex["beta"], atol=0)
    r1 = rows[(0, 1)]
    for key in ("log_s_base", "log_s_rescue"):
        np.testing.assert_allclose(np.exp(r1[key] - r1[key].max()), ex["row1_ratio"], rtol=1e-12)
    assert _ids(r1["final"]) == ex["row1_final_tau_0.15"]
    _, _, _, _, rows16 = _case_rows(case, 0.16, 0.16)
    assert _ids(rows16[(0, 1)]["final"]) == ex["row1_final_tau_0.16"]


def test_fractional_beta_case():
    """Sec. 3.1 Eq. beta and Sec. 3.2 Eq. rescue_score with 0 < beta < 1."""
    case = _load("fractional_beta_case.json")
    ex = case["expected"]
    C, R, beta, rq, rows = _case_rows(case)
    np.testing.assert_allclose(R[0], ex["radii"], atol=1e-15)
    np.testing.assert_allclose(rq[0], [ex["r_low"], ex["r_high"]], rtol=1e-14)
    np.testing.assert_allclose(beta[0], ex["beta"], rtol=1e-12, atol=1e-15)
    r4 = rows[(0, 4)]
    np.testing.assert_allclose(np.exp(r4["log_s_base"] - r4["log_s_base"].max()), ex["row4_base_ratio"], rtol=1e-12)
    np.testing.assert_allclose(np.exp(r4["log_s_rescue"] - r4["log_s_rescue"].max()), ex["row4_rescue_ratio"], rtol=1e-12)
    assert _ids(r4["final"]) == ex["row4_final"]


@pytest.mark.parametrize("idx", [0, 1])
def test_quantiles_and_beta_hand_computed(idx):
    """Sec. 3.1: r_low / r_high are the 0.5 / 0.9 quantiles; Eq. beta."""
    case = _load("quantiles.json")["cases"][idx]
    R = np.array(case["radii"], dtype=np.float64)[None]
    beta, rq = oracle.rescue_coefficients(R)
    np.testing.assert_allclose(rq[0], [case["r_low"], case["r_high"]], rtol=1e-14)
    np.testing.assert_allclose(beta[0], case["beta"], rtol=1e-12, atol=1e-15)


def test_quantile_matches_library_linear_rule():
    """The type-7 reading equals numpy's default ('linear') quantile."""
    rng = np.random.default_rng(3)
    for n in (1, 2, 3, 7, 64, 1000, 1023):
        x = rng.lognormal(0, 0.7, size=n)
        for p in (0.5, 0.9):
            assert oracle.quantile_type7(x, p) == pytest.approx(np.quantile(x, p), rel=1e-14, abs=0)


# ------------------------------------------------------------ geometry (Sec. 2.4, App. E)

def test_full_l2_bound_holds_for_every_key():
    """Sec. 2.4 Eq. full_l2_bound: max_k q.k <= q.c_b + |q| r_b, unattenuated."""
    rng = np.random.default_rng(7)
    d, B, N = 16, 8, 8 * 9 + 5
    scales = np.repeat(rng.lognormal(0, 1.0, size=-(-N // B)), B)[:N]
    K = rng.standard_normal((1, N, d)) * scales[None, :, None] + rng.standard_normal(d)
    C, R = oracle.block_stats(K, B)
    Qs = rng.standard_normal((50, d)) * 3
    for b, (s, e) in enumerate(oracle.block_ranges(N, B)):
        logits = Qs @ K[0, s:e].T
        bound = Qs @ C[0, b] + np.linalg.norm(Qs, axis=1) * R[0, b]
        assert (logits.max(axis=1) <= bound + 1e-10).all()
        # The key that defines the radius, queried along its own deviation,
        # meets the bound exactly (the ball is tight).
        far = int(np.argmax(np.linalg.norm(K[0, s:e] - C[0, b], axis=1)))
        u = K[0, s + far] - C[0, b]
        assert u @ K[0, s + far] == pytest.approx(u @ C[0, b] + np.linalg.norm(u) * R[0, b], rel=1e-12)


def test_attenuated_score_is_not_a_bound():
    """App. E: K = {-u, u}, q = u gives c = 0, r = 1, max logit 1, rescue logit beta."""
    u = np.array([0.6, 0.8, 0.0])
    K = np.stack([-u, u])[None]
    C, R = oracle.block_stats(K, 2)
    np.testing.assert_allclose(C[0, 0], 0, atol=1e-15)
    assert R[0, 0] == pytest.approx(1.0, rel=1e-15)
    for b in (0.0, 0.3, 1.0):
        lb, lr = oracle.branch_logits(u[None], C[0], R[0], np.array([b]), 1)
        assert lb[0, 0] == pytest.approx(0.0, abs=1e-15)
        assert lr[0, 0] == pytest.approx(b, rel=1e-14, abs=1e-15)
        assert (lr[0, 0] < (K[0] @ u).max()) == (b < 1.0)


def _box_bound(q, K):
    lo, hi = K.min(axis=0), K.max(axis=0)
    return np.maximum(q * lo, q * hi).sum()


def test_l2_ball_versus_coordinate_box_examples():
    """App. E, Eq. quest_box: neither bound dominates (two 2-D examples)."""
    e1, e2 = np.eye(2)
    K = np.stack([e1, -e1, e2, -e2])
    C, R = oracle.block_stats(K[None], 4)
    q = np.array([1.0, 1.0])
    assert q @ C[0, 0] + np.linalg.norm(q) * R[0, 0] == pytest.approx(math.sqrt(2), rel=1e-15)
    assert _box_bound(q, K) == pytest.approx(2.0)
    eps = 0.25
    K = np.stack([e1, -e1, eps * e2, -eps * e2])
    C, R = oracle.block_stats(K[None], 4)
    q = e2
    assert R[0, 0] == pytest.approx(1.0, rel=1e-15)
    assert q @ C[0, 0] + np.linalg.norm(q) * R[0, 0] == pytest.approx(1.0, rel=1e-15)
    assert _box_bound(q, K) == pytest.approx(eps)


def test_translation_and_rotation_invariance():
    """App. E: q.c_b and r_b are unchanged under a common orthogonal map; a
    common shift moves c_b and leaves r_b unchanged."""
    rng = np.random.default_rng(11)
    d, B, N = 12, 5, 23
    K = rng.standard_normal((1, N, d)) * 2
    q = rng.standard_normal(d)
    C, R = oracle.block_stats(K, B)
    Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
    C2, R2 = oracle.block_stats(K @ Qm.T, B)
    np.testing.assert_allclose(R2, R, rtol=1e-12)
    np.testing.assert_allclose(C2[0] @ (Qm @ q), C[0] @ q, rtol=1e-10, atol=1e-12)
    shift = rng.standard_normal(d) * 5
    C3, R3 = oracle.block_stats(K + shift, B)
    np.testing.assert_allclose(R3, R, rtol=1e-10)
    np.testing.assert_allclose(C3, C + shift, rtol=1e-12, atol=1e-12)


def test_partial_last_block_uses_its_own_count():
    """Sec. 3.1: c_b divides by |K_b|; a last block of one key has r = 0."""
    K = np.arange(5 * 3, dtype=np.float64).reshape(1, 5, 3)
    C, R = oracle.block_stats(K, 4)
    np.testing.assert_allclose(C[0, 0], K[0, :4].mean(axis=0))
    np.testing.assert_allclose(C[0, 1], K[0, 4])
    assert R[0, 1] == 0.0


# ------------------------------------------------------------ scoring / selection

def _random_case(seed=0, d=8, B=4, N=4 * 7 + 2, Hq=4, Hkv=2):
    rng = np.random.default_rng(seed)
    scales = np.repeat(rng.lognormal(0, 0.8, size=-(-N // B)), B)[:N]
    K = rng.standard_normal((Hkv, N, d)) * scales[None, :, None] + 2 * rng.standard_normal((Hkv, 1, d))
    Q = rng.standard_normal((Hq, N, d)) * 1.5
    C, R = oracle.block_stats(K, B)
    beta, _ = oracle.rescue_coefficients(R)
    return Q, K, C, R, beta, B


def test_rescue_logit_dominates_base_and_equals_l2_bound_at_beta_one():
    """Sec. 3.2: l_rescue >= l_base; with beta = 1 it equals U^L2."""
    Q, K, C, R, beta, B = _random_case()
    lb, lr = oracle.branch_logits(Q[0, :B], C[0], R[0], beta[0], C.shape[1])
    assert (lr >= lb).all()
    lb1, lr1 = oracle.branch_logits(Q[0, :B], C[0], R[0], np.ones_like(beta[0]), C.shape[1])
    bound = Q[0, :B] @ C[0].T + np.linalg.norm(Q[0, :B], axis=1)[:, None] * R[0][None, :]
    np.testing.assert_allclose(lr1, bound, rtol=1e-13)


def test_shift_choice_does_not_change_masks():
    """Sec. 3.2: the shared shift cancels; per-block log-sum-exp gives the same
    relative scores and masks."""
    Q, K, C, R, beta, B = _random_case(seed=5)
    M = C.shape[1]
    for i in range(M):
        s, e = i * B, min((i + 1) * B, Q.shape[1])
        lb, lr = oracle.branch_logits(Q[1, s:e], C[0], R[0], beta[0], i + 1)
        ref_b, ref_r = oracle.branch_log_scores(Q[1, s:e], C[0], R[0], beta[0], i + 1)
        for logits, ref in ((lb, ref_b), (lr, ref_r)):
            x = logits / math.sqrt(Q.shape[2])
            col_max = x.max(axis=0)
            lse = col_max + np.log(np.exp(x - col_max).sum(axis=0))
            np.testing.assert_allclose(lse - lse.max(), ref - ref.max(), atol=1e-12)


def test_brute_force_scores_on_tiny_input():
    """Eq. base_score / rescue_score / block_aggregation by explicit loops."""
    Q, K, C, R, beta, B = _random_case(seed=9, d=3, B=3, N=10, Hq=1, Hkv=1)
    i = 3
    toks = range(i * B, min((i + 1) * B, Q.shape[1]))
    S_b, S_r = [], []
    for b in range(i + 1):
        sb = sr = 0.0
        for t in toks:
            dot = sum(Q[0, t, j] * C[0, b, j] for j in range(3))
            nq = math.sqrt(sum(Q[0, t, j] ** 2 for j in range(3)))
            sb += math.exp(dot / math.sqrt(3))
            sr += math.exp((dot + nq * R[0, b] * beta[0, b]) / math.sqrt(3))
        S_b.append(sb)
        S_r.append(sr)
    lb, lr = oracle.branch_log_scores(Q[0, list(toks)], C[0], R[0], beta[0], i + 1)
    np.testing.assert_allclose(lb - lb.max(), np.log(S_b) - max(np.log(S_b)), atol=1e-12)
    np.testing.assert_allclose(lr - lr.max(), np.log(S_r) - max(np.log(S_r)), atol=1e-12)


def test_threshold_monotonicity():
    """App. E / Sec. 3.2: lowering a threshold cannot shrink its branch's mask."""
    Q, K, C, R, beta, B = _random_case(seed=2)
    taus = [1.0, 0.95, 0.8, 0.5, 0.2, 0.05, 0.0]
    prev = None
    for t in taus:
        rows = oracle.select(Q, C, R, beta, B, t, t, 0, 1, 0)
        cur = {k: (v["base"], v["rescue"]) for k, v in rows.items()}
        if prev is not None:
            for k in cur:
                assert (cur[k][0] >= prev[k][0]).all() and (cur[k][1] >= prev[k][1]).all()
        prev = cur


def test_alpha_one_keeps_argmax_and_alpha_zero_keeps_all():
    """Eq. branch_thresholds special cases."""
    Q, K, C, R, beta, B = _random_case(seed=4)
    rows = oracle.select(Q, C, R, beta, B, 1.0, 1.0, 0, 1, 0)
    for (h, i), r in rows.items():
        assert _ids(r["base"]) == [int(np.argmax(r["log_s_base"]))]
        assert _ids(r["rescue"]) == [int(np.argmax(r["log_s_rescue"]))]
    rows = oracle.select(Q, C, R, beta, B, 0.0, 0.0, 0, 1, 0)
    for (h, i), r in rows.items():
        assert r["final"].all() and r["final"].shape == (i + 1,)


def test_ties_are_all_kept():
    """Eq. branch_thresholds is inclusive: zero queries tie every candidate."""
    Q, K, C, R, beta, B = _random_case(seed=8)
    Q[:, :2 * B] = 0.0
    rows = oracle.select(Q, C, R, beta, B, 0.99, 0.99, 0, 1, 0, rows=[(0, 1), (3, 1)])
    for r in rows.values():
        assert r["base"].all() and r["rescue"].all()


@pytest.mark.parametrize("sink,local,recent", [(1, 2, 0), (0, 1, 0), (2, 3, 1), (1, 1, 2)])
def test_forced_blocks_always_present(sink, local, recent):
    """Sec. 3.2 union with forced sink, local-window and recent blocks."""
    Q, K, C, R, beta, B = _random_case(seed=6)
    M = C.shape[1]
    rows = oracle.select(Q, C, R, beta, B, 1.0, 1.0, sink, local, recent)
    for (h, i), r in rows.items():
        f = r["final"]
        assert f[:min(sink, i + 1)].all()
        assert f[max(0, i - local + 1):i + 1].all()
        if i >= M - recent:
            assert f.all()


def test_union_differs_from_both_branches_in_needle_case():
    """Sec. 3.2 / App. E: rescue-only selection can drop base-selected blocks."""
    case = _load("needle_case.json")
    _, _, _, _, rows = _case_rows(case)
    r = rows[(0, 2)]
    assert not (r["base"] <= r["rescue"]).all()
    assert (r["final"] != r["base"]).any() and (r["final"] != r["rescue"]).any()


# ------------------------------------------------------------ attention (Eq. (1), Sec. 3.3)

def test_full_selection_equals_brute_force_dense_attention():
    """alpha = 0 keeps every causal block, so sparse attention reduces to the
    dense causal softmax attention of Eq. (1), computed here by brute force."""
    rng = np.random.default_rng(1)
    d, B, N = 8, 4, 4 * 5 + 3
    Q, K, V = (rng.standard_normal((N, d)) for _ in range(3))
    C, R = oracle.block_stats(K[None], B)
    beta, _ = oracle.rescue_coefficients(R)
    rows = oracle.select(Q[None], C, R, beta, B, 0.0, 0.0, 0, 1, 0)
    lists = {i: _ids(rows[(0, i)]["final"]) for i in range(C.shape[1])}
    sparse = np.concatenate([oracle.attention_on_mask(Q, K, V, B, lists)[i] for i in sorted(lists)])
    brute = np.zeros((N, d))
    for t in range(N):
        w = [math.exp(sum(Q[t, j] * K[s, j] for j in range(d)) / math.sqrt(d)) for s in range(t + 1)]
        z = sum(w)
        for s in range(t + 1):
            brute[t] += w[s] / z * V[s]
    np.testing.assert_allclose(sparse, brute, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(oracle.dense_causal_attention(Q, K, V), brute, rtol=1e-11, atol=1e-12)


def test_attention_invariances():
    """Softmax over retained keys: a constant added to every key leaves the
    output unchanged; the output is linear in V; one retained key returns its
    value; a query with no retained causal key gets zeros."""
    rng = np.random.default_rng(12)
    d, B, N = 6, 4, 16
    Q, K, V, V2 = (rng.standard_normal((N, d)) for _ in range(4))
    lists = {0: [0], 1: [0, 1], 2: [1, 2], 3: [0, 3]}
    o1 = oracle.attention_on_mask(Q, K, V, B, lists)
    o2 = oracle.attention_on_mask(Q, K + rng.standard_normal(d), V, B, lists)
    for i in lists:
        np.testing.assert_allclose(o1[i], o2[i], rtol=1e-11, atol=1e-12)
    a, b = 0.7, -1.3
    o3 = oracle.attention_on_mask(Q, K, a * V + b * V2, B, lists)
    o4 = oracle.attention_on_mask(Q, K, V2, B, lists)
    for i in lists:
        np.testing.assert_allclose(o3[i], a * o1[i] + b * o4[i], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(o1[0][0], V[0], rtol=1e-14)
    assert not oracle.attention_rows(Q, K, V, B, 2, [3]).any()


def test_density_counts_selected_pairs_once():
    """Sec. 4.4 Eq. actual_density on hand-counted rows."""
    rows = [np.array([True]), np.array([True, False]), np.array([True, False, True])]
    assert oracle.density(rows) == pytest.approx(4 / 6)
    assert oracle.density([np.ones(k, bool) for k in range(1, 9)]) == 1.0


def test_list_mask_roundtrip():
    rows = {(0, 0): np.array([True]), (0, 2): np.array([True, False, True]), (1, 1): np.array([False, True])}
    counts, idx = oracle.lists_from_masks(rows, 2, 3)
    back = oracle.masks_from_lists(counts, idx, rows.keys())
    for k in rows:
        assert (back[k] == rows[k]).all()


# ------------------------------------------------ supporting selectors (Table selector_ablation)

def _variant_scores(K_block, q, variant):
    """Unscaled logit of one query against one block, through the oracle."""
    K = np.asarray(K_block, dtype=np.float64)[None]
    C, R = oracle.block_stats(K, K.shape[1])
    Vc, Hw = oracle.block_box(K, K.shape[1])
    return oracle.variant_logits(np.asarray(q, dtype=np.float64)[None], C[0], R[0], Vc[0], Hw[0], 1, variant)[0, 0]


def test_variant_logits_on_the_appendix_examples():
    """App. geometry: K = {e1, -e1, e2, -e2}, q = (1, 1): full-L2 sqrt 2, box 2;
    K = {e1, -e1, eps e2, -eps e2}, q = e2: full-L2 1, box eps; centroid 0 in both."""
    e1, e2 = np.eye(2)
    K = np.stack([e1, -e1, e2, -e2])
    q = np.array([1.0, 1.0])
    assert _variant_scores(K, q, "full_l2") == pytest.approx(math.sqrt(2), rel=1e-15)
    assert _variant_scores(K, q, "box") == pytest.approx(2.0, rel=1e-15)
    assert _variant_scores(K, q, "centroid") == pytest.approx(0.0, abs=1e-15)
    eps = 0.25
    K = np.stack([e1, -e1, eps * e2, -eps * e2])
    assert _variant_scores(K, e2, "full_l2") == pytest.approx(1.0, rel=1e-15)
    assert _variant_scores(K, e2, "box") == pytest.approx(eps, rel=1e-15)


def test_box_and_full_l2_dominate_every_token_logit():
    """Both are upper bounds of max_k q.k over the block (App. geometry); the box
    is attained when the block holds its own extreme corner."""
    rng = np.random.default_rng(21)
    for _ in range(50):
        K = rng.standard_normal((7, 5)) * rng.uniform(0.1, 3.0)
        q = rng.standard_normal(5)
        top = (K @ q).max()
        assert _variant_scores(K, q, "box") >= top - 1e-12
        assert _variant_scores(K, q, "full_l2") >= top - 1e-12
        assert _variant_scores(K, q, "centroid") <= top + 1e-12
    lo, hi = np.array([-1.0, 0.5, -2.0]), np.array([2.0, 1.5, -1.0])
    q = np.array([1.0, -1.0, 2.0])
    corner = np.where(q >= 0, hi, lo)
    K = np.stack([lo, hi, corner])
    assert _variant_scores(K, q, "box") == pytest.approx(q @ corner, rel=1e-15)


def test_single_key_blocks_reduce_every_variant_to_the_token_logit():
    rng = np.random.default_rng(22)
    k, q = rng.standard_normal(6), rng.standard_normal(6)
    for v in oracle.SELECTOR_VARIANTS:
        assert _variant_scores(k[None], q, v) == pytest.approx(q @ k, rel=1e-12)


def test_rotation_keeps_centroid_and_l2_scores_but_not_the_box():
    """App. geometry: centroid dot product and radius are invariant under a common
    orthogonal transform; the coordinate-wise box is not."""
    e1, e2 = np.eye(2)
    K = np.stack([e1, -e1, e2, -e2])
    q = np.array([1.0, 1.0])
    c, s = math.cos(math.pi / 4), math.sin(math.pi / 4)
    Rot = np.array([[c, -s], [s, c]])
    for v in ("centroid", "full_l2"):
        assert _variant_scores(K @ Rot.T, Rot @ q, v) == pytest.approx(_variant_scores(K, q, v), abs=1e-12)
    assert _variant_scores(K @ Rot.T, Rot @ q, "box") != pytest.approx(_variant_scores(K, q, "box"), abs=1e-3)


def test_budget_selection_fractions():
    """Fixed budget: rho = 1 keeps all, a tiny rho keeps the argmax (ties too),
    and a larger budget never drops a block."""
    log_s = np.log(np.array([0.2, 0.9, 0.1, 0.9, 0.5, 0.05]))
    assert oracle.top_fraction(log_s, 1.0)[0].all()
    m, _ = oracle.top_fraction(log_s, 1e-6)
    assert m.tolist() == [False, True, False, True, False, False]
    prev = np.zeros(6, bool)
    for rho in (0.1, 0.3, 0.5, 0.7, 0.9, 1.0):
        m, margin = oracle.top_fraction(log_s, rho)
        assert m.sum() >= math.ceil(rho * 6)
        assert (m | ~prev).all() and (m == (margin >= 0)).all()
        prev = m


def test_variant_rows_keep_forced_blocks_and_threshold_extremes():
    rng = np.random.default_rng(23)
    d, B, N = 8, 4, 40
    Q = rng.standard_normal((1, N, d))
    K = rng.standard_normal((1, N, d))
    C, R = oracle.block_stats(K, B)
    Vc, Hw = oracle.block_box(K, B)
    M = N // B
    for v, param in (("centroid", 0.5), ("full_l2", 0.5), ("box", 0.2)):
        rows = oracle.select_variant(Q, C, R, Vc, Hw, B, v, param, 1, 2, 0)
        for (h, i), r in rows.items():
            assert (r["final"][r["forced"]]).all() and r["final"][0] and r["final"][i]
            assert (r["final"] == (r["branch"] | r["forced"])).all()
    for v in ("centroid", "full_l2"):
        all_rows = oracle.select_variant(Q, C, R, Vc, Hw, B, v, 0.0, 0, 1, 0)
        assert all(r["final"].all() for r in all_rows.values())
        top_rows = oracle.select_variant(Q, C, R, Vc, Hw, B, v, 1.0, 0, 1, 0)
        for r in top_rows.values():
            assert r["branch"].sum() == 1 and r["branch"][np.argmax(r["log_s"])]
    box_all = oracle.select_variant(Q, C, R, Vc, Hw, B, "box", 1.0, 0, 1, 0)
    assert all(r["final"].all() for r in box_all.values())
    assert len(box_all) == M


def test_variant_aggregation_sums_scaled_exponentials_over_tokens():
    """Sec. 3.2 Eq. block_aggregation applied to the supporting selectors of
    Table selector_ablation (centroid, Eq. full_l2_bound, Eq. quest_box): each
    block score sums exp(logit / sqrt d) over the query block's tokens.  Two
    different queries make the sum, the max over tokens and the mean logit
    disagree, and d = 4 makes the 1/sqrt(d) scale matter (tests/golden)."""
    case = _load("variant_aggregation_case.json")
    ex = case["expected"]
    B = case["block_size"]
    K = np.array(case["keys"], dtype=np.float64)[None]
    Q = np.array(case["queries"], dtype=np.float64)[None]
    C, R = oracle.block_stats(K, B)
    Vc, Hw = oracle.block_box(K, B)
    np.testing.assert_allclose(C[0], ex["centroids"], atol=1e-15)
    np.testing.assert_allclose(R[0], ex["radii"], atol=1e-15)
    np.testing.assert_allclose(Vc[0], ex["box_center"], atol=1e-15)
    np.testing.assert_allclose(Hw[0], ex["box_half"], atol=1e-15)
    Qi = Q[0, B:2 * B]
    for variant, ratio in ex["row1_ratio"].items():
        log_s = oracle.variant_log_scores(Qi, C[0], R[0], Vc[0], Hw[0], 2, variant)
        assert log_s[0] - log_s[1] == pytest.approx(math.log(ratio), abs=1e-12), variant
    M = K.shape[1] // B
    for key, final in ex["row1_final"].items():
        variant, param = key.rsplit("_", 1)
        row = oracle.select_variant_row(Qi, C[0], R[0], Vc[0], Hw[0], 1, M, variant, float(param),
                                        case["n_sink"], case["n_local"], case["n_recent"])
        assert _ids(row["final"]) == final, key


# ---------------------------------------------------------------- batches
# App. "Additional A100 System Measurements", prompt throughput: batched
# prompts are independent causal sequences, none concatenated into another.

def _batch(lengths, H_q=2, H_kv=1, d=8, seed=0, noise=None):
    rng = np.random.default_rng(seed)
    T = sum(lengths)
    Q = rng.standard_normal((H_q, T, d))
    K = rng.standard_normal((H_kv, T, d)) + 2.0
    if noise is not None:  # per-sequence key spread, so radius distributions differ
        off = oracle.batch_offsets(lengths)
        for s, sc in enumerate(noise):
            K[:, off[s]:off[s + 1]] = 2.0 + sc * rng.standard_normal((H_kv, lengths[s], d)) * \
                rng.lognormal(0.0, 0.7, size=(H_kv, lengths[s], 1))
    V = rng.standard_normal((H_kv, T, d))
    return Q, K, V


def _all_rows(result):
    return {s: {h: {i: np.nonzero(r["final"])[0].tolist() for (hh, i), r in rows.items() if hh == h}
                for h in sorted({hh for (hh, _) in rows})}
            for s, rows in result.items()}


def test_batch_of_one_is_the_single_sequence():
    Q, K, V = _batch([75])
    C, R = oracle.block_stats(K, 16)
    beta, rq = oracle.rescue_coefficients(R)
    Cb, Rb, betab, rqb = oracle.batch_block_stats(K, [75], 16)
    assert np.array_equal(C, Cb) and np.array_equal(R, Rb) and np.array_equal(beta, betab)
    assert np.array_equal(rq, rqb[0])
    single = oracle.select(Q, C, R, beta, 16, 0.9, 0.95, 1, 1, 0)
    batched = oracle.batch_select(Q, K, [75], 16, 0.9, 0.95, 1, 1, 0)[0]
    assert single.keys() == batched.keys()
    assert all(np.array_equal(single[k]["final"], batched[k]["final"]) for k in single)


def test_batch_sequences_are_independent():
    lengths = [50, 70, 33]
    Q, K, V = _batch(lengths, seed=1)
    Q2, K2, V2 = Q.copy(), K.copy(), V.copy()
    off = oracle.batch_offsets(lengths)
    rng = np.random.default_rng(9)
    for X in (Q2, K2, V2):  # change sequence 1 only
        X[:, off[1]:off[2]] += rng.standard_normal(X[:, off[1]:off[2]].shape)
    a = oracle.batch_select(Q, K, lengths, 16, 0.9, 0.95, 1, 1, 0)
    b = oracle.batch_select(Q2, K2, lengths, 16, 0.9, 0.95, 1, 1, 0)
    oa = oracle.batch_attention_on_mask(Q, K, V, lengths, 16, _all_rows(a))
    ob = oracle.batch_attention_on_mask(Q2, K2, V2, lengths, 16, _all_rows(a))
    for s in (0, 2):
        for k in a[s]:
            assert np.array_equal(a[s][k]["log_s_base"], b[s][k]["log_s_base"])
            assert np.array_equal(a[s][k]["final"], b[s][k]["final"])
        for h in oa[s]:
            for i in oa[s][h]:
                assert np.array_equal(oa[s][h][i], ob[s][h][i])
    assert any(not np.array_equal(a[1][k]["log_s_base"], b[1][k]["log_s_base"]) for k in a[1])
    Ma = oracle.batch_block_stats(K, lengths, 16)
    Mb = oracle.batch_block_stats(K2, lengths, 16)
    m = [0] + list(np.cumsum([-(-n // 16) for n in lengths]))
    for s in (0, 2):
        assert np.array_equal(Ma[1][:, m[s]:m[s + 1]], Mb[1][:, m[s]:m[s + 1]])
        assert np.array_equal(Ma[3][s], Mb[3][s])


def test_batch_at_full_selection_is_each_sequence_dense_attention():
    lengths = [40, 29, 57]
    Q, K, V = _batch(lengths, H_q=2, H_kv=1, seed=2)
    sel = oracle.batch_select(Q, K, lengths, 16, 0.0, 0.0, 0, 1, 0)
    for s, rows in sel.items():
        for (h, i), r in rows.items():
            assert r["final"].all()  # alpha = 0 keeps every causal block
    out = oracle.batch_attention_on_mask(Q, K, V, lengths, 16, _all_rows(sel))
    Qs, Ks, Vs = (oracle.batch_sequences(X, lengths) for X in (Q, K, V))
    off = oracle.batch_offsets(lengths)
    for s in range(len(lengths)):
        for h in range(2):
            got = np.concatenate([out[s][h][i] for i in sorted(out[s][h])])
            assert np.allclose(got, oracle.dense_causal_attention(Qs[s][h], Ks[s][0], Vs[s][0]), atol=1e-12)
            if s > 0:  # the concatenated sequence would also attend to earlier prompts
                cat = oracle.dense_causal_attention(Q[h, :off[s + 1]], K[0, :off[s + 1]], V[0, :off[s + 1]])
                assert not np.allclose(got, cat[off[s]:])


def test_block_aligned_batch_shares_centroids_but_not_beta_with_the_concatenation():
    lengths = [64, 96, 48]
    _, K, _ = _batch(lengths, H_q=1, H_kv=1, seed=3, noise=[0.3, 1.0, 3.0])
    Cb, Rb, betab, rqb = oracle.batch_block_stats(K, lengths, 16)
    Cc, Rc = oracle.block_stats(K, 16)
    assert np.array_equal(Cb, Cc) and np.array_equal(Rb, Rc)   # same block partition
    beta_cat, _ = oracle.rescue_coefficients(Rc)
    assert not np.allclose(betab, beta_cat)                    # per-prompt quantiles differ
    off = [0, 4, 10, 13]
    for s in range(3):
        beta_s, rq_s = oracle.rescue_coefficients(Rc[:, off[s]:off[s + 1]])
        assert np.array_equal(betab[:, off[s]:off[s + 1]], beta_s) and np.array_equal(rqb[s], rq_s)


# ---------------------------------------------------------------- FP8 E4M3
# Values fixed by the OCP 8-bit floating-point format definition of E4M3
# (bias 7, 3 mantissa bits, subnormals m/8 * 2^-6, largest finite 448).

@pytest.mark.parametrize("x,code", [
    (0.0, 0x00), (-0.0, 0x80), (1.0, 0x38), (-1.0, 0xb8), (448.0, 0x7e), (-448.0, 0xfe),
    (2.0 ** -6, 0x08), (2.0 ** -9, 0x01), (7 * 2.0 ** -9, 0x07), (1.75, 0x3e), (240.0, 0x77),
    (1.0625, 0x38),            # tie between 1.0 (mantissa 0) and 1.125 (1): even
    (1.1875, 0x3a),            # tie between 1.125 (1) and 1.25 (2): even
    (2.0 ** -10, 0x00),        # tie between 0 and the smallest subnormal: even
    (3 * 2.0 ** -10, 0x02),    # tie between 2^-9 (1) and 2^-8 (2): even
    (464.0, 0x7e), (1e6, 0x7e), (-1e6, 0xfe),   # saturation
    (1.06, 0x38), (1.07, 0x39),
])
def test_e4m3_format_values(x, code):
    assert int(oracle.e4m3_encode(np.array([x]))[0]) == code
    exact = {0.0, 1.0, 448.0, 2.0 ** -6, 2.0 ** -9, 7 * 2.0 ** -9, 1.75, 240.0}
    if abs(x) in exact:  # representable values decode back to themselves, sign included
        v = oracle.e4m3_decode(np.array([code]))[0]
        assert v == x and np.signbit(v) == np.signbit(x)


def test_e4m3_codes_round_trip_in_order():
    codes = np.arange(256, dtype=np.uint8)
    v = oracle.e4m3_decode(codes)
    finite = ~np.isnan(v)
    assert finite.sum() == 254 and np.isnan(v[0x7f]) and np.isnan(v[0xff])
    assert np.array_equal(oracle.e4m3_encode(v[finite]), codes[finite])
    pos = v[:0x7f]
    assert np.all(np.diff(pos) > 0) and pos[-1] == 448.0


def test_e4m3_rounds_to_nearest_with_ties_to_even():
    grid = oracle.e4m3_decode(np.arange(0x7f, dtype=np.uint8))   # 0 .. 448, code = index
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.uniform(0, 448, 4000), rng.uniform(0, 2.0 ** -5, 2000),
                        (grid[:-1] + grid[1:]) / 2])            # every midpoint is a tie
    got = oracle.e4m3_encode(x).astype(np.int64)
    d = np.abs(grid[None, :] - x[:, None])
    best = d.min(axis=1)
    for k in range(len(x)):
        cands = np.nonzero(d[k] == best[k])[0]
        want = cands[0] if len(cands) == 1 else [c for c in cands if c % 2 == 0][0]
        assert got[k] == want, (x[k], got[k], want)


def test_fp8_quantize_maps_amax_to_448():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((3, 50, 8)) * np.array([0.01, 1.0, 300.0])[:, None, None]
    amax = oracle.fp8_amax(X)
    assert np.allclose(amax, np.abs(X).reshape(3, -1).max(axis=1))
    codes, deq = oracle.fp8_quantize(X, amax)
    for h in range(3):
        i = np.unravel_index(np.abs(X[h]).argmax(), X[h].shape)
        assert codes[h][i] & 0x7f == 0x7e                      # the largest magnitude becomes 448
    Y = oracle.fp8_dequantize(codes, deq)
    # Relative error of a normal E4M3 value is at most 2^-4 (3 mantissa bits, nearest).
    big = np.abs(X) >= 2.0 ** -6 * deq[:, None, None] * 1.01
    assert np.all(np.abs(Y - X)[big] <= 2.0 ** -4 * np.abs(X)[big] * 1.0001)
