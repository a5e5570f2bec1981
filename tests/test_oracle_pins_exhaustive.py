"""Exhaustive pins of the oracle's coverage budgets and allocator at n <= 64,
and a hand-computed case of the clustered-summary certificate.

Coverage: the paper's coverage definition (the smallest k whose top-k mass
reaches the retained fraction) and its lemma that top-k selection is
coverage-optimal (no other set of the same size holds more mass).  All 2^n
subsets are enumerated for n <= 20; for 20 < n <= 64 every single swap of a
kept key for an evicted one is checked, which by the exchange argument of the
lemma certifies that no k-subset beats the top-k set.

Allocation: the appendix's exact-budget protocol (sum b_h = B_real,
b_h in [b_min, n-1]); an exact dynamic program over the heads gives the true
minimum of sum_h c_h(b_h), which the heuristic can only match or exceed, and
matches on convex curves, for n up to 64.

Certificate: the appendix theorem on clustered tail summaries, evaluated by
hand on two clusters chosen so that every quantity is a short fraction.
"""
import math

import numpy as np
import pytest

import oracle


# --------------------------------------------------------------------------
# Coverage: all subsets for n <= 20.

def _subset_masses(a):
    """Mass and size of every subset of range(n), indexed by its bit mask."""
    n = len(a)
    mass = np.zeros(1 << n, np.float64)
    size = np.zeros(1 << n, np.int8)
    for i in range(n):
        lo, hi = 1 << i, 1 << (i + 1)
        mass[lo:hi] = mass[:lo] + a[i]
        size[lo:hi] = size[:lo] + 1
    return mass, size


def _best_by_size(mass, size, n):
    best = np.full(n + 1, -1.0)
    np.maximum.at(best, size.astype(np.int64), mass)
    return best


@pytest.mark.parametrize("n", [14, 17, 20])
def test_coverage_all_subsets(n):
    rng = np.random.default_rng(100 + n)
    for trial in range(4):
        s = (rng.random(n) ** 3).astype(np.float32)
        if trial == 1:
            s[::3] = s[1]          # ties
        if trial == 2:
            s[:4] = 0.0            # zero mass keys
        a = oracle.normalize(s)
        perm = oracle.order(s)
        mass, size = _subset_masses(a)
        best = _best_by_size(mass, size, n)
        prefix = np.concatenate([[0.0], np.cumsum(a[perm])])
        # the lemma: for every size k the top-k set holds the most mass
        np.testing.assert_allclose(best, prefix, rtol=1e-12, atol=1e-15)
        # k_eta is the smallest size reaching the target, for targets away
        # from every prefix mass (so that summation order cannot decide)
        for retain in rng.uniform(0.05, 0.999, 12):
            if np.min(np.abs(prefix - retain)) < 1e-9:
                continue
            k = oracle.coverage(s, perm, float(retain))
            assert best[k] >= retain and (k == 1 or best[k - 1] < retain), (n, retain, k)


# --------------------------------------------------------------------------
# Coverage: every pairwise swap for 20 < n <= 64.

@pytest.mark.parametrize("n", [21, 33, 48, 64])
def test_coverage_pairwise_swaps(n):
    rng = np.random.default_rng(200 + n)
    for trial in range(6):
        s = (rng.gamma(0.3, size=n)).astype(np.float32)
        if trial % 2:
            s[rng.integers(0, n, n // 3)] = s[0]   # ties
        a = oracle.normalize(s)
        perm = oracle.order(s)
        for retain in (0.3, 0.6, 0.9, 0.99):
            k = oracle.coverage(s, perm, retain)
            kept = np.zeros(n, bool)
            kept[perm[:k]] = True
            top = a[kept].sum()
            assert top >= retain - 1e-15
            # minimality: the top-(k-1) set misses the target
            assert k == 1 or a[perm[:k - 1]].sum() < retain
            # no single swap (i kept, j evicted) gains mass: every swapped set
            # has mass top - a_i + a_j <= top
            gain = a[~kept][None, :] - a[kept][:, None]
            assert (gain <= 0.0).all(), (n, retain, float(gain.max()))
            # ties are broken toward the lower position among equal scores
            if k < n:
                worst_kept = perm[k - 1]
                for j in np.flatnonzero(~kept):
                    if s[j] == s[worst_kept]:
                        assert j > worst_kept


# --------------------------------------------------------------------------
# Allocation against an exact dynamic program, n up to 64.

def _dp_optimum(c, B_real, b_min):
    """min sum_h c_h(b_h) subject to sum_h b_h = B_real, b_min <= b_h <= n-1
    (fp64 sums of the fp32 curve values), by a DP over heads."""
    H, n = c.shape
    cand = np.arange(b_min, n)
    best = np.full(B_real + 1, np.inf)
    best[0] = 0.0
    for h in range(H):
        nxt = np.full(B_real + 1, np.inf)
        vals = c[h, cand].astype(np.float64)
        for t in np.flatnonzero(np.isfinite(best)):
            tt = t + cand
            ok = tt <= B_real
            np.minimum.at(nxt, tt[ok], best[t] + vals[ok])
        best = nxt
    return best[B_real]


def _random_curves(rng, H, n):
    c = np.abs(np.cumsum(rng.standard_normal((H, n)), axis=1))[:, ::-1]
    return np.ascontiguousarray(c * rng.uniform(0.1, 10, (H, 1))).astype(np.float32)


@pytest.mark.parametrize("n", [32, 48, 64])
def test_allocate_vs_exact_dp_up_to_64(n):
    rng = np.random.default_rng(300 + n)
    x = np.arange(n, dtype=np.float64)
    for trial in range(8):
        H = int(rng.integers(2, 5))
        n_keep = int(rng.integers(2, n + 1))
        br, bm = oracle.budget_params(H, n, n_keep)
        c = _random_curves(rng, H, n)
        b, _ = oracle.allocate(c, n_keep)
        assert b.sum() == br and b.min() >= bm and b.max() <= n - 1
        obj = sum(float(c[h, b[h]]) for h in range(H))
        opt = _dp_optimum(c, br, bm)
        assert opt <= obj + 1e-9 * max(1.0, abs(obj))
        # convex decreasing curves: the Lagrangian allocation with its
        # best-marginal repair reaches the optimum
        cc = np.stack([rng.uniform(0.5, 4) * (n - x) ** 2 / n + rng.uniform(0, 1)
                       for _ in range(H)]).astype(np.float32)
        b2, _ = oracle.allocate(cc, n_keep)
        obj2 = sum(float(cc[h, b2[h]]) for h in range(H))
        assert obj2 == pytest.approx(_dp_optimum(cc, br, bm), rel=1e-9, abs=1e-9)


def test_dp_reference_on_a_hand_case():
    # the DP itself, on a case small enough to solve by hand: two heads,
    # b in {1, 2, 3}, B_real = 4: the options (1,3), (2,2), (3,1) cost
    # 9 + 1, 4 + 5, 2 + 6, so the optimum is 8 at (3, 1); with B_real = 3
    # only (1, 2) and (2, 1) remain: 9 + 5 and 4 + 6, optimum 10
    c = np.array([[99, 9, 4, 2], [99, 6, 5, 1]], np.float32)
    assert _dp_optimum(c, 4, 1) == 8.0
    assert _dp_optimum(c, 3, 1) == 10.0


# --------------------------------------------------------------------------
# The clustered-summary certificate on a hand-computed case.

def test_cluster_certificate_hand_computed():
    # d = 2, query q = (1, 0), scale = ln 1.25, one kept row (key 0, value
    # (1, 0)) and two clusters:
    #   g = 1: n = 2, mean key (ln 2 / ln 1.25, 0) so lbar = ln 2 and
    #          Zhat_1 = 2 * 2 = 4; key radius 1 so r = ln 1.25, e^r = 5/4;
    #          mean value (0, 3), value radius 1
    #   g = 2: n = 3, mean key (-ln 2 / ln 1.25, 0) so Zhat_2 = 3 / 2;
    #          key radius 0; mean value (-2, 0), value radius 1/2
    # Then Zhat = 1 + 4 + 3/2 = 13/2 and
    #   D_Z = (5/4 - 1)(5/4) 4 + 0 = 5/4
    #   D_N = (5/4) 4 ((1/4) 3 + 1) + 1 (3/2)(0 + 1/2) = 35/4 + 3/4 = 19/2
    #   V'  = max(|(1,0)|, 3 + 1, 2 + 1/2) = 4
    #   D_Z <= Zhat / 3 holds (5/4 <= 13/6), so the bound is
    #   3 / Zhat (D_N + V' D_Z) = (6/13)(19/2 + 5) = 87/13
    #   Ohat = ((1, 0) + 4 (0, 3) + (3/2)(-2, 0)) / Zhat = (-4/13, 24/13)
    #   structural form: 3 (1 - p_S) max_g e^{r_g} (2 V' (e^{r_g} - 1) + rho_g)
    #   with p_S = 2/13: 3 (11/13) max(5/4 (2 4 (1/4) + 1), 1 (0 + 1/2))
    #   = (33/13)(15/4) = 495/52
    a = math.log(2.0) / math.log(1.25)
    cl = dict(kbar=np.array([[a, 0.0], [-a, 0.0]]), vbar=np.array([[0.0, 3.0], [-2.0, 0.0]]),
              count=np.array([2, 3], np.int32), R=np.array([1.0, 0.0], np.float32),
              rho=np.array([1.0, 0.5], np.float32), vmax_kept=1.0)
    out, c = oracle.cluster_estimate(np.array([1.0, 0.0]), np.zeros((1, 2)),
                                     np.array([[1.0, 0.0]]), cl, math.log(1.25))
    np.testing.assert_allclose(out, [-4.0 / 13.0, 24.0 / 13.0], rtol=1e-12)
    assert c["lse"] == pytest.approx(math.log(6.5), rel=1e-12)
    assert c["dz"] == pytest.approx((5.0 / 4.0) / 6.5, rel=1e-12)
    assert c["dn"] == pytest.approx((19.0 / 2.0) / 6.5, rel=1e-12)
    assert c["vmax"] == 4.0
    assert c["bound"] == pytest.approx(87.0 / 13.0, rel=1e-12)
    assert c["structural"] == pytest.approx(495.0 / 52.0, rel=1e-12)
    # a wider key radius on cluster 1 breaks the condition D_Z <= Zhat / 3:
    # at R_1 = ln 2 / ln 1.25, e^r = 2 and D_Z = (2 - 1) 2 4 = 8 > 13/6
    cl["R"] = np.array([a, 0.0], np.float32)
    _, c2 = oracle.cluster_estimate(np.array([1.0, 0.0]), np.zeros((1, 2)),
                                    np.array([[1.0, 0.0]]), cl, math.log(1.25))
    assert c2["dz"] > 1.0 / 3.0 and math.isinf(c2["bound"])
