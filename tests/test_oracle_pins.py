"""Pins of the fp64 CPU oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  The pins are chosen so that a
plausible slip in the oracle (a dropped term, a flipped sign, an off-by-one
rank, a transposed operand, a wrong tie rule) fails at least one of them.
None of these tests touch the GPU path.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.stats import norm

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# Scores: Section 3 one-row setup (softmax of <q,k>/sqrt(d)) and the window
# scorer (sum of softmax weights over window rows).

def test_scores_closed_form_single_row():
    # logits (0, ln 2, ln 3) give softmax (1/6, 1/3, 1/2).  d = 4 so the
    # 1/sqrt(d) = 1/2 scale is exercised: keys carry 2*logit in coordinate 0.
    d = 4
    q = np.array([[1.0, 0.0, 0.0, 0.0]])
    lg = np.array([0.0, math.log(2.0), math.log(3.0)])
    k = np.zeros((3, d))
    k[:, 0] = 2.0 * lg
    k[:, 1] = [5.0, -7.0, 3.0]  # orthogonal to q: must not matter
    s = oracle.scores(q, [2], k, 1.0 / math.sqrt(d), causal=True)
    np.testing.assert_allclose(s, [1 / 6, 1 / 3, 1 / 2], rtol=0, atol=1e-15)


def test_scores_operand_roles_not_symmetric():
    # q . k with q = (1, 0) and k_j = (0, l_j): all logits 0 -> uniform.  A
    # transposed or swapped operand would read the second coordinate.
    q = np.array([[1.0, 0.0]])
    k = np.array([[0.0, 3.0], [0.0, -1.0], [0.0, 9.0]])
    s = oracle.scores(q, [2], k, 1.0, causal=True)
    np.testing.assert_allclose(s, [1 / 3] * 3, atol=1e-15)


def test_scores_causal_rows_and_row_sum():
    # Two rows at positions 0 and 2 over n = 3 keys.  Row at position 0 sees
    # only key 0 (weight 1); row at position 2 sees all three.
    q = np.array([[1.0], [1.0]])
    k = np.array([[0.0], [math.log(2.0)], [math.log(3.0)]])
    s = oracle.scores(q, [0, 2], k, 1.0, causal=True)
    np.testing.assert_allclose(s, [1 + 1 / 6, 1 / 3, 1 / 2], atol=1e-15)
    s_nc = oracle.scores(q, [0, 2], k, 1.0, causal=False)
    np.testing.assert_allclose(s_nc, [2 / 6, 4 / 6, 1.0], atol=1e-15)


def test_scores_sum_equals_number_of_rows():
    # Each softmax row sums to one, so sum_j s_j = number of window rows.
    rng = np.random.default_rng(0)
    n, d, M = 300, 16, 12
    q = rng.standard_normal((M, d))
    k = rng.standard_normal((n, d)) * 2.0
    qpos = n - 4 + (np.arange(M) % 4)
    s, lse = oracle.scores(q, qpos, k, 1 / math.sqrt(d), causal=True, with_lse=True)
    assert abs(s.sum() - M) < 1e-12 * M
    assert (s > 0).all()
    # keys after the last visible position get nothing
    assert s[n - 1] > 0 and s[: n - 4].min() > 0
    # lse of a row = log sum exp of its logits (brute force on row 0)
    lg = (k[: qpos[0] + 1] @ q[0]) / math.sqrt(d)
    assert abs(lse[0] - (lg.max() + math.log(np.exp(lg - lg.max()).sum()))) < 1e-12


# --------------------------------------------------------------------------
# Ordering: score descending, ties by index (Section 3 ordering pi; Algorithm 1).

def test_order_flat_row_keeps_lowest_indices():
    # Flat-row proposition (appendix "Tightness on flat rows"): on A_j = 1/n a
    # weight-only rule with index tie-breaking keeps the first k indices.
    n = 50
    s = np.full(n, 1.0 / n, np.float32)
    perm = oracle.order(s)
    assert perm.tolist() == list(range(n))
    assert oracle.select(perm, 7).tolist() == list(range(7))


@pytest.mark.parametrize("n", [1, 2, 5, 7])
def test_order_exhaustive_small(n):
    # Every assignment of values from {0, 1, 2} (with ties) to n <= 7 keys:
    # rank(i) < rank(j) iff s_i > s_j or (s_i == s_j and i < j).
    vals = [0.0, 0.5, 2.0]
    for combo in itertools.product(vals, repeat=n) if n <= 5 else [
            tuple(np.random.default_rng(n).choice(vals, n)) for _ in range(200)]:
        s = np.array(combo, np.float32)
        perm = oracle.order(s)
        rank = np.empty(n, int)
        rank[perm] = np.arange(n)
        for i in range(n):
            for j in range(n):
                if i != j:
                    before = s[i] > s[j] or (s[i] == s[j] and i < j)
                    assert (rank[i] < rank[j]) == before


@pytest.mark.parametrize("n,w", [(1, 1), (4, 2), (5, 5), (7, 3)])
def test_order_keep_window_exhaustive_small(n, w):
    # The keep-window order ranks the last w positions first as if their
    # scores were +infinity: with t_j = +inf for the window and s_j otherwise,
    # rank(i) < rank(j) iff t_i > t_j or (t_i == t_j and i < j), for every
    # assignment of tied values.
    vals = [0.0, 0.5, 2.0]
    for combo in itertools.product(vals, repeat=n) if n <= 5 else [
            tuple(np.random.default_rng(n).choice(vals, n)) for _ in range(200)]:
        s = np.array(combo, np.float32)
        perm = oracle.order(s, keep_window=w)
        t = s.astype(np.float64)
        t[n - w:] = np.inf
        rank = np.empty(n, int)
        rank[perm] = np.arange(n)
        for i in range(n):
            for j in range(n):
                if i != j:
                    before = t[i] > t[j] or (t[i] == t[j] and i < j)
                    assert (rank[i] < rank[j]) == before
    # keep_window = 0 is the plain order
    s = np.random.default_rng(3).random(n).astype(np.float32)
    assert np.array_equal(oracle.order(s, keep_window=0), oracle.order(s))


def test_normalize_clips_and_sums_to_one():
    # appendix "CertKV: implementation": a = (s)_+ / sum (s)_+
    s = np.array([2.0, -1.0, 1.0, 0.0, 1.0], np.float32)
    a = oracle.normalize(s)
    np.testing.assert_allclose(a, [0.5, 0.0, 0.25, 0.0, 0.25], atol=0)
    np.testing.assert_allclose(oracle.normalize(np.zeros(4, np.float32)), [0.25] * 4)


# --------------------------------------------------------------------------
# Curves: Section 4.1 Eq. certkv-curve; appendix suffix moments and the
# identity c^2 = (m Q - |W|^2)_+ = m S.

def _direct_curve(a, perm, v, b):
    """c(b) from the centered definition: m * sqrt(E_r |v - v*|^2)."""
    E = perm[b:]
    m = a[E].sum()
    vstar = (a[E, None] * v[E]).sum(0) / m
    S = (a[E] * ((v[E] - vstar) ** 2).sum(1)).sum()
    return m * math.sqrt(S / m), m, S


def test_curve_matches_centered_definition():
    rng = np.random.default_rng(1)
    n, d = 64, 5
    s = rng.random(n).astype(np.float32) + 0.01
    v = rng.standard_normal((n, d)) * rng.uniform(0.2, 3.0, (n, 1))
    perm = oracle.order(s)
    a = oracle.normalize(s)
    c, c32 = oracle.curves(s, perm, v)
    for b in range(n):
        ref, m, S = _direct_curve(a, perm, v, b)
        assert abs(c[b] - ref) <= 1e-12 * (1 + ref), b
        assert abs(c[b] ** 2 - m * S) <= 1e-12 * (1 + m * S)
    assert c[n - 1] == pytest.approx(0.0, abs=1e-7)
    np.testing.assert_array_equal(c32, c.astype(np.float32))


def test_curve_two_point_witness():
    # Theorem "exact envelopes" (Section 'Why centered dispersion'): a tail of
    # two equal-weight points v* +/- delta u has S = m delta^2, c = m delta.
    delta = 0.75
    vstar = np.array([1.0, -2.0, 0.5])
    u = np.array([0.0, 0.6, 0.8])  # unit vector
    v = np.stack([np.array([9.0, 9.0, 9.0]), vstar + delta * u, vstar - delta * u])
    s = np.array([0.5, 0.25, 0.25], np.float32)  # key 0 ranks first
    perm = oracle.order(s)
    assert perm.tolist() == [0, 1, 2]
    c, _ = oracle.curves(s, perm, v)
    m = 0.5
    assert c[1] == pytest.approx(m * delta, rel=1e-12)
    assert c[2] == pytest.approx(0.0, abs=1e-8)  # one-point tail
    # c(0): whole set; closed form m=1, centroid, second moment by hand
    mean = 0.5 * v[0] + 0.25 * v[1] + 0.25 * v[2]
    S0 = 0.5 * ((v[0] - mean) ** 2).sum() + 0.25 * ((v[1] - mean) ** 2).sum() + \
        0.25 * ((v[2] - mean) ** 2).sum()
    assert c[0] == pytest.approx(math.sqrt(S0), rel=1e-12)


def test_curve_constant_values_is_zero_and_scale():
    # Equal values leave nothing to disperse: c == 0.  Scaling v by k scales c
    # by |k| (c is a norm-type statistic).
    n, d = 20, 3
    s = np.linspace(1.0, 2.0, n).astype(np.float32)
    perm = oracle.order(s)
    c, _ = oracle.curves(s, perm, np.tile([1.0, 2.0, -3.0], (n, 1)))
    assert np.abs(c).max() < 1e-6
    rng = np.random.default_rng(3)
    v = rng.standard_normal((n, d))
    c1, _ = oracle.curves(s, perm, v)
    c2, _ = oracle.curves(s, perm, -3.0 * v)
    np.testing.assert_allclose(c2, 3.0 * c1, rtol=1e-10, atol=1e-7)  # c(n-1) is sqrt of a rounding residue


def test_curve_uses_rank_order_not_position_order():
    # Scores reversed relative to positions: the evicted suffix at b = n-1 is
    # position 0 (the lowest score), so c(n-2) involves positions 0 and 1.
    v = np.array([[0.0], [2.0], [100.0]])
    s = np.array([1.0, 2.0, 3.0], np.float32)
    perm = oracle.order(s)
    assert perm.tolist() == [2, 1, 0]
    c, _ = oracle.curves(s, perm, v)
    a = s.astype(np.float64) / float(s.astype(np.float64).sum())
    m = a[0] + a[1]
    vs = (a[0] * 0.0 + a[1] * 2.0) / m
    S = a[0] * vs ** 2 + a[1] * (2.0 - vs) ** 2
    assert c[1] == pytest.approx(math.sqrt(m * S), rel=1e-12)


# --------------------------------------------------------------------------
# Allocation: exact slot accounting (Section 4.1) and Algorithm 1.

def test_budget_algebra():
    br, bm = oracle.budget_params(8, 32768, 3277, 0.2)
    assert br == 8 * 3277 - 8 and bm == max(1, math.floor(0.2 * br / 8))
    assert oracle.budget_params(4, 1024, 129, 0.2) == (512, 25)
    with pytest.raises(oracle.OracleError):
        oracle.budget_params(4, 1024, 1, 0.2)  # n_keep >= 2
    with pytest.raises(oracle.OracleError):
        oracle.budget_params(4, 1024, 1025, 0.2)  # n_keep <= n


def _random_curves(rng, H, n):
    c = np.abs(np.cumsum(rng.standard_normal((H, n)), axis=1))[:, ::-1]
    return np.ascontiguousarray(c * rng.uniform(0.1, 10, (H, 1))).astype(np.float32)


def test_allocate_exact_sum_and_bounds():
    rng = np.random.default_rng(4)
    for trial in range(40):
        H = int(rng.integers(1, 9))
        n = int(rng.integers(4, 200))
        n_keep = int(rng.integers(2, n + 1))
        c = _random_curves(rng, H, n)
        b, _ = oracle.allocate(c, n_keep)
        br, bm = oracle.budget_params(H, n, n_keep)
        assert b.sum() == br
        assert (b >= bm).all() and (b <= n - 1).all()


def test_allocate_keep_all():
    # n_keep = n: B_real = H (n-1) forces b_h = n-1 for every head.
    rng = np.random.default_rng(5)
    c = _random_curves(rng, 6, 40)
    b, _ = oracle.allocate(c, 40)
    assert b.tolist() == [39] * 6


def test_initial_multiplier_selects_b_min():
    # At lambda_hi = 2 max c + 1 the penalty dominates: every head's argmin over
    # [b_min, n-1] is b_min, so sum b(lambda_hi) <= B_real holds at the start.
    rng = np.random.default_rng(6)
    c = _random_curves(rng, 5, 120)
    lam = 2.0 * float(c.astype(np.float64).max()) + 1.0
    for h in range(5):
        assert oracle.argmin_penalized(c[h], 7, 119, lam) == 7
    # argmin ties go to the smallest b
    flat = np.zeros(10, np.float32)
    assert oracle.argmin_penalized(flat, 2, 9, 0.0) == 2


def _dp_optimum(c, B_real, b_min):
    H, n = c.shape
    INF = float("inf")
    best = {0: 0.0}
    for h in range(H):
        nxt = {}
        for tot, val in best.items():
            for b in range(b_min, n):
                t = tot + b
                if t > B_real:
                    break
                v = val + float(c[h, b])
                if v < nxt.get(t, INF):
                    nxt[t] = v
        best = nxt
    return best[B_real]


def test_allocate_vs_exact_dp():
    # The exact DP optimum never exceeds the heuristic's objective; on convex
    # curves the Lagrangian + marginal repair reaches it.
    rng = np.random.default_rng(7)
    for trial in range(25):
        H, n = int(rng.integers(2, 4)), int(rng.integers(6, 25))
        n_keep = int(rng.integers(2, n + 1))
        br, bm = oracle.budget_params(H, n, n_keep)
        c = _random_curves(rng, H, n)
        b, _ = oracle.allocate(c, n_keep)
        obj = sum(float(c[h, b[h]]) for h in range(H))
        assert _dp_optimum(c, br, bm) <= obj + 1e-9
        # convex decreasing curves: c(b) = scale * (n - b)^2 / n + offset
        x = np.arange(n, dtype=np.float64)
        cc = np.stack([rng.uniform(0.5, 4) * (n - x) ** 2 / n + rng.uniform(0, 1)
                       for _ in range(H)]).astype(np.float32)
        b2, _ = oracle.allocate(cc, n_keep)
        obj2 = sum(float(cc[h, b2[h]]) for h in range(H))
        assert obj2 == pytest.approx(_dp_optimum(cc, br, bm), rel=1e-9, abs=1e-9)


def test_bisection_trajectory_on_linear_curves():
    # Linear curves c_h(b) = kappa_h (n-1-b): c + lambda b is minimized at n-1
    # when lambda < kappa_h and at b_min otherwise (ties -> b_min).  With
    # B_real = b_min + n - 1 the total drops to B_real exactly at lambda = 1,
    # so lambda_hi must settle on 1 from above, within one bisection interval
    # of the initial lambda_hi = 2 max c + 1, and stay a dyadic multiple of it.
    n, T = 41, 40
    x = (n - 1 - np.arange(n)).astype(np.float64)
    c = np.stack([1.0 * x, 3.0 * x]).astype(np.float32)
    for n_keep in range(2, n + 1):
        br, bm = oracle.budget_params(2, n, n_keep)
        if br == bm + n - 1:
            break
    else:
        pytest.fail("no n_keep with B_real = b_min + n - 1")
    b, rep, (lo, hi) = oracle.allocate(c, n_keep, steps=T, with_lambda=True)
    lam0 = 2.0 * float(c.max()) + 1.0
    assert 1.0 <= hi <= 1.0 + lam0 / 2 ** T
    assert lo < 1.0
    ratio = hi * 2 ** T / lam0
    assert ratio == math.floor(ratio)
    assert b.tolist() == [bm, n - 1] and rep == 0


def test_repair_alone_reaches_optimum_on_convex_curves():
    # With T = 0 the allocation is b(lambda_hi) = b_min everywhere followed by
    # best-marginal repair; on convex curves that greedy is optimal.
    rng = np.random.default_rng(17)
    for trial in range(20):
        H, n = int(rng.integers(2, 4)), int(rng.integers(6, 25))
        n_keep = int(rng.integers(2, n + 1))
        br, bm = oracle.budget_params(H, n, n_keep)
        x = np.arange(n, dtype=np.float64)
        cc = np.stack([rng.uniform(0.5, 4) * (n - x) ** 2 / n for _ in range(H)]
                      ).astype(np.float32)
        b, rep = oracle.allocate(cc, n_keep, steps=0)
        assert rep == br - H * bm
        obj = sum(float(cc[h, b[h]]) for h in range(H))
        assert obj == pytest.approx(_dp_optimum(cc, br, bm), rel=1e-9, abs=1e-9)


def test_allocate_prefers_dispersed_head():
    # Two heads, identical except head 1's values are 10x more dispersed: the
    # budget must shift toward head 1 (a head with more tail dispersion gets
    # more slots, Section 4.1).
    rng = np.random.default_rng(8)
    n, d = 256, 8
    s = rng.random(n).astype(np.float32)
    perm = oracle.order(s)
    v = rng.standard_normal((n, d))
    _, c0 = oracle.curves(s, perm, v)
    _, c1 = oracle.curves(s, perm, 10.0 * v)
    b, _ = oracle.allocate(np.stack([c0, c1]), 40)
    assert b[1] > b[0]


# --------------------------------------------------------------------------
# Selection and coverage (Section 3 Eq. coverage-def; lemma "top-k is
# coverage-optimal"; fact "order-statistic mass bound").

def test_select_partition_and_topk():
    rng = np.random.default_rng(9)
    n = 500
    s = rng.random(n).astype(np.float32)
    s[::7] = s[3]  # ties
    perm = oracle.order(s)
    for b in [1, 13, 250, 499]:
        kept = oracle.select(perm, b)
        assert kept.tolist() == sorted(kept.tolist())
        ev = np.setdiff1d(np.arange(n), kept)
        assert len(kept) + len(ev) == n and len(np.intersect1d(kept, ev)) == 0
        assert len(kept) == b
        # every kept key outranks every evicted key
        lowest_kept = min(kept, key=lambda j: (-s[j], j))
        for j in ev:
            assert (s[lowest_kept], -lowest_kept) > (s[j], -j) or \
                (s[lowest_kept] > s[j]) or (s[lowest_kept] == s[j] and lowest_kept < j)


def test_coverage_minimal_and_subset_optimal():
    # Brute force over all subsets (n <= 12): no set smaller than k_eta reaches
    # the retained mass, and the top-k_eta set does.
    rng = np.random.default_rng(10)
    for trial in range(30):
        n = int(rng.integers(1, 13))
        s = (rng.random(n) ** 3).astype(np.float32)
        retain = float(rng.uniform(0.05, 0.99))
        perm = oracle.order(s)
        k = oracle.coverage(s, perm, retain)
        a = oracle.normalize(s)
        assert a[perm[:k]].sum() >= retain - 1e-15
        best_smaller = 0.0
        for size in range(1, k):
            for sub in itertools.combinations(range(n), size):
                best_smaller = max(best_smaller, a[list(sub)].sum())
        assert best_smaller < retain


def test_coverage_threshold_is_inclusive():
    # Eq. coverage-def uses >=: a = (1/2, 1/4, 1/4) reaches 3/4 at k = 2.
    s = np.array([0.5, 0.25, 0.25], np.float32)
    perm = oracle.order(s)
    assert oracle.coverage(s, perm, 0.75) == 2
    assert oracle.coverage(s, perm, 0.5) == 1
    assert oracle.coverage(s, perm, 1.0) == 3


def test_coverage_floor_counts_from_k_min():
    # With a floor k_min the budget is the smallest k >= k_min reaching the
    # retained mass: the definition's k when that is already >= k_min.
    rng = np.random.default_rng(12)
    for trial in range(50):
        n = int(rng.integers(2, 40))
        s = (rng.random(n) ** 3).astype(np.float32)
        perm = oracle.order(s)
        a = oracle.normalize(s)
        retain = float(rng.uniform(0.05, 0.99))
        k1 = oracle.coverage(s, perm, retain)
        k_min = int(rng.integers(1, n + 1))
        k = oracle.coverage(s, perm, retain, k_min=k_min)
        assert k == max(k1, k_min)
        assert a[perm[:k]].sum() >= retain - 1e-15


def test_order_statistic_mass_bound():
    # 1 - p(k) <= (n - k)/(k + 1) for every row and k in [n-1].
    rng = np.random.default_rng(11)
    for trial in range(20):
        n = int(rng.integers(2, 200))
        s = np.exp(rng.standard_normal(n) * rng.uniform(0, 4)).astype(np.float32)
        perm = oracle.order(s)
        a = oracle.normalize(s)
        p = np.cumsum(a[perm])
        for k in range(1, n):
            assert 1 - p[k - 1] <= (n - k) / (k + 1) + 1e-12


def test_gaussian_coverage_law():
    # Section 3.1: for i.i.d. N(0, sigma^2) logits, K_eta/n ->
    # Phi(Phi^{-1}(1-eta) - sigma), about 0.61 at sigma = 1, eta = 0.1.
    g = golden("coverage_law.json")
    n = 200_000
    rng = np.random.default_rng(12)
    z = rng.standard_normal(n) * g["sigma"]
    s = oracle.scores(np.array([[1.0]]), [n - 1], z[:, None], 1.0, causal=True)
    s32 = s.astype(np.float32)
    k = oracle.coverage(s32, oracle.order(s32), 1.0 - g["eta"])
    law = norm.cdf(norm.ppf(1 - g["eta"]) - g["sigma"])
    assert round(law, 2) == g["kept_fraction"]
    assert abs(k / n - law) < 0.01


# --------------------------------------------------------------------------
# Tail summary: Section 4.1 centroids; Theorem "fixed-row tail
# factorization" (the unique correction is the weighted tail sum).

def test_tail_pooled_reconstruction_exact():
    rng = np.random.default_rng(13)
    n, d = 300, 6
    s = rng.random(n).astype(np.float32) + 0.01
    kmat = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    perm = oracle.order(s)
    kept = oracle.select(perm, 40)
    ks, vs, m = oracle.tail(s, kept, kmat, v)
    a = oracle.normalize(s)
    mask = np.zeros(n, bool)
    mask[kept] = True
    assert m == pytest.approx(a[~mask].sum(), rel=1e-14)
    full = (a[:, None] * v).sum(0)
    recon = (a[mask, None] * v[mask]).sum(0) + m * vs
    np.testing.assert_allclose(recon, full, rtol=0, atol=1e-13)
    fullk = (a[:, None] * kmat).sum(0)
    np.testing.assert_allclose((a[mask, None] * kmat[mask]).sum(0) + m * ks, fullk,
                               atol=1e-13)
    # the helper agrees: compensated error with u = m v* is zero
    assert oracle.row_error(a, v, mask, m * vs) < 1e-13


def test_tail_fixed_row_factorization_per_row():
    # For one realized row, scoring with that row's weights makes the slot the
    # exact tail aggregate u* = sum_T A_j V_j: O_S + m v* = O.
    A = np.array([0.5, 0.25, 0.125, 0.0625, 0.0625])
    V = np.array([[1.0, 0.0], [0.0, 2.0], [-4.0, 1.0], [3.0, 3.0], [0.5, -8.0]])
    s = A.astype(np.float32)
    kept = oracle.select(oracle.order(s), 2)
    assert kept.tolist() == [0, 1]
    _, vs, m = oracle.tail(s, kept, V, V)
    assert m == 0.25
    mask = np.zeros(5, bool)
    mask[kept] = True
    assert oracle.row_error(A, V, mask, m * vs) == 0.0
    # without the slot the error is |u*| (the truncated scheme)
    ustar = (A[2:, None] * V[2:]).sum(0)
    assert oracle.row_error(A, V, mask) == pytest.approx(np.linalg.norm(ustar), rel=1e-15)


def test_tail_keep_all_but_one_and_empty_mass():
    n, d = 10, 3
    rng = np.random.default_rng(14)
    s = rng.random(n).astype(np.float32) + 0.1
    kmat, v = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    perm = oracle.order(s)
    kept = oracle.select(perm, n - 1)
    ks, vs, m = oracle.tail(s, kept, kmat, v)
    last = perm[-1]
    np.testing.assert_allclose(ks, kmat[last], rtol=1e-14)
    np.testing.assert_allclose(vs, v[last], rtol=1e-14)
    # zero-score evicted keys: m = 0 and the slot is the zero vector
    s0 = s.copy()
    s0[last] = 0.0
    ks0, vs0, m0 = oracle.tail(s0, kept, kmat, v)
    assert m0 == 0.0 and not ks0.any() and not vs0.any()


# --------------------------------------------------------------------------
# The paper's worked examples (golden fixtures).

def test_worked_example_oracle_subset_witness():
    g = golden("worked_examples.json")["oracle_subset_witness"]
    A, V = np.array(g["A"]), np.array(g["V"], float)
    np.testing.assert_allclose((A[:, None] * V).sum(0), g["O"], atol=1e-15)
    assert oracle.row_error(A, V, [1, 1, 0, 0]) == pytest.approx(g["E_keep_1_2"], abs=1e-15)
    assert oracle.row_error(A, V, [0, 0, 1, 1]) == pytest.approx(g["E_keep_3_4"], abs=1e-15)
    # top-2 by weight is {1,2} in the paper's 1-based labels
    assert oracle.select(oracle.order(np.float32(A)), 2).tolist() == [0, 1]


def test_worked_example_proxy_separation():
    g = golden("worked_examples.json")["proxy_separation"]
    A, V, Vh = np.array(g["A"]), np.array(g["V"], float), g["Vhat"]
    s_unc = (A * np.abs(V)).astype(np.float32)
    s_cen = (A * np.abs(V - Vh)).astype(np.float32)
    np.testing.assert_allclose(s_unc, g["s_uncentered"], rtol=1e-6)
    np.testing.assert_allclose(s_cen, g["s_centered"], rtol=1e-6)
    S_unc = oracle.select(oracle.order(s_unc), 2)
    S_cen = oracle.select(oracle.order(s_cen), 2)
    assert S_unc.tolist() == g["top2_uncentered"] and S_cen.tolist() == g["top2_centered"]
    for S, want in [(S_unc, g["compensated_error_uncentered"]),
                    (S_cen, g["compensated_error_centered"])]:
        mask = np.zeros(4, bool)
        mask[S] = True
        u = np.array([A[~mask].sum() * Vh])
        assert oracle.row_error(A, V, mask, u) == pytest.approx(want, rel=1e-14)


def test_worked_example_one_swap():
    g = golden("worked_examples.json")["one_swap_counterexample"]
    A, U = np.array(g["A"]), np.array(g["u"], float)
    V = 4.0 * U

    def E(keep):
        mask = np.zeros(4, bool)
        mask[list(keep)] = True
        return oracle.row_error(A, V, mask)

    assert E([0, 1]) == pytest.approx(g["E_keep_1_2"], rel=1e-14)
    assert E([2, 3]) == pytest.approx(g["E_keep_3_4"], rel=1e-14)
    sw = {k: eval(v, {"sqrt": math.sqrt}) for k, v in g["one_swaps"].items()}
    assert E([0, 2]) == pytest.approx(sw["keep_1_3"], rel=1e-14)
    assert E([0, 3]) == pytest.approx(sw["keep_1_4"], rel=1e-14)
    assert E([1, 2]) == pytest.approx(sw["keep_2_3"], rel=1e-14)
    assert E([1, 3]) == pytest.approx(sw["keep_2_4"], rel=1e-14)


def test_physical_cache_bytes():
    # Appendix "Physical cache capacity": 8.59 GB full -> 0.86 GB packed at 64K
    # and 10x.  Per (layer, sequence) the packed cache holds sum_h (b_h + 1) =
    # B_real + H = H * n_keep rows, n_keep = floor(n (1 - r)).
    g = golden("physical_cache.json")
    sh = g["model_shape"]
    n, H = g["context"], sh["kv_heads"]
    n_keep = math.floor(n * (1 - g["evicted_fraction"]) + 1e-9)
    rng = np.random.default_rng(15)
    c = _random_curves(rng, H, n)
    b, _ = oracle.allocate(c, n_keep)
    rows = int((b + 1).sum())
    assert rows == H * n_keep
    row_bytes = sh["head_dim"] * sh["bytes_per_elem"] * 2  # K and V
    packed = sh["layers"] * rows * row_bytes
    full = sh["layers"] * H * n * row_bytes
    assert round(packed / 1e9, 2) == g["certkv_cache_GB"]
    assert round(full / 1e9, 2) == g["full_cache_GB"]


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -8 + 2 ** -20,
                  3.0e38, 0.0], np.float32)
    bits = oracle.f32_to_bf16_bits(x)
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F81, 0x7F62, 0x0000]


# --------------------------------------------------------------------------
# One block end to end: invariants that hold at any size.

def test_compress_block_invariants():
    rng = np.random.default_rng(16)
    n, H, G, d, w = 400, 3, 2, 8, 6
    q = rng.standard_normal((w, H * G, d))
    k = rng.standard_normal((n, H, d))
    v = rng.standard_normal((n, H, d))
    n_keep = 41
    out = oracle.compress_block(q, k, v, n_keep, 1 / math.sqrt(d))
    br, bm = oracle.budget_params(H, n, n_keep)
    np.testing.assert_allclose(out["s"].sum(1), w * G, rtol=1e-12)
    assert out["budgets"].sum() == br
    for h in range(H):
        kept = out["kept"][h]
        assert len(kept) == out["budgets"][h]
        ks, vs, m = oracle.tail(out["s32"][h], kept, k[:, h], v[:, h])
        np.testing.assert_allclose(out["v_star"][h], vs, rtol=1e-15)
        assert out["tail_mass"][h] == m
        # scores of one head match the single-head scorer
        qh = q[:, h * G:(h + 1) * G].reshape(w * G, d)
        qpos = np.repeat(n - w + np.arange(w), G)
        np.testing.assert_allclose(out["s"][h], oracle.scores(qh, qpos, k[:, h], 1 / math.sqrt(d)),
                                   rtol=1e-14)


def test_compress_block_keep_window():
    # Every head keeps the w window keys; the budget algebra is unchanged; a
    # budget too small to hold the window is infeasible.
    rng = np.random.default_rng(17)
    n, H, G, d, w = 400, 3, 2, 8, 6
    q = rng.standard_normal((w, H * G, d))
    k = rng.standard_normal((n, H, d))
    v = rng.standard_normal((n, H, d))
    n_keep = 41
    out = oracle.compress_block(q, k, v, n_keep, 1 / math.sqrt(d), keep_window=True)
    plain = oracle.compress_block(q, k, v, n_keep, 1 / math.sqrt(d))
    br, bm = oracle.budget_params(H, n, n_keep)
    assert bm >= w and out["budgets"].sum() == br
    np.testing.assert_array_equal(out["s"], plain["s"])
    for h in range(H):
        assert out["perm"][h, :w].tolist() == list(range(n - w, n))
        assert set(range(n - w, n)) <= set(out["kept"][h].tolist())
        # ranks after the window follow the plain order of the other keys
        rest = [j for j in plain["perm"][h] if j < n - w]
        assert out["perm"][h, w:].tolist() == rest
    with pytest.raises(oracle.OracleError) as e:
        oracle.compress_block(q, k, v, 6, 1 / math.sqrt(d), keep_window=True)  # b_min = 1 < w
    assert e.value.code == oracle.ORA_EINFEASIBLE


# --------------------------------------------------------------------------
# The one-token repair (Algorithm 1: "repair one token at a time") as a
# selection problem.  Greedy: repeatedly take the head whose next marginal
# d = c(b+1) - c(b) is smallest, ties to the lowest head.  Claim used by the
# GPU allocator: the greedy consumes elements in increasing order of the key
# (running max of the head's marginals up to that element, head, position).
# Checked here against the oracle's sequential repair on random curves.

def _keyed_repair(c, start, R):
    H, n = c.shape
    keys = []
    for h in range(H):
        run = -math.inf
        for i in range(int(start[h]), n - 1):
            run = max(run, float(c[h, i + 1]) - float(c[h, i]))
            keys.append((run, h, i))
    keys.sort()
    b = np.array(start, dtype=np.int64)
    for _, h, _ in keys[:R]:
        b[h] += 1
    return b


def test_repair_equals_running_max_key_order():
    rng = np.random.default_rng(18)
    for trial in range(300):
        H, n = int(rng.integers(1, 6)), int(rng.integers(3, 30))
        n_keep = int(rng.integers(2, n + 1))
        # few distinct levels so that ties between heads and within runs occur
        c = rng.integers(0, 4, (H, n)).astype(np.float32) * 0.5
        if trial % 3 == 0:
            c = np.sort(c, axis=1)[:, ::-1].copy()
        br, bm = oracle.budget_params(H, n, n_keep)
        b_seq, rep = oracle.allocate(c, n_keep, steps=0)  # start = b_min everywhere
        start = np.full(H, bm)
        R = br - H * bm
        assert rep == R
        assert _keyed_repair(c, start, R).tolist() == b_seq.tolist()
