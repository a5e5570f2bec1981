"""CPU pins of the oracle's one-factor ablation branches (appendix, one-factor
ablations table): the tail-mass and uncentered statistics, the uniform and
greedy-marginal allocators and the no-slot budget algebra."""
import itertools

import numpy as np
import pytest

import oracle


def _rank(rng, n):
    s = rng.gamma(0.4, size=n).astype(np.float32)
    return s, oracle.order(s)


def test_tail_mass_is_the_evicted_share_of_the_weights():
    n = 40
    s = np.full(n, 0.7, np.float32)              # equal scores: a = 1/n
    perm = oracle.order(s)
    v = np.random.default_rng(0).normal(size=(n, 8))
    c, _ = oracle.curves(s, perm, v, "tail_mass")
    np.testing.assert_allclose(c, (n - np.arange(n)) / n, rtol=1e-14)
    s, perm = _rank(np.random.default_rng(1), 300)
    c, _ = oracle.curves(s, perm, np.zeros((300, 4)), "tail_mass")
    assert abs(c[0] - 1.0) <= 1e-14              # every weight evicted at b = 0
    assert np.all(np.diff(c) <= 0)               # one more key kept, less mass


def test_identical_values_have_no_centered_dispersion():
    rng = np.random.default_rng(2)
    n, d = 200, 16
    s, perm = _rank(rng, n)
    v0 = rng.normal(size=d)
    v = np.tile(v0, (n, 1))
    cc, _ = oracle.curves(s, perm, v, "centered")
    cu, _ = oracle.curves(s, perm, v, "uncentered")
    cm, _ = oracle.curves(s, perm, v, "tail_mass")
    assert np.max(cc) <= 1e-6 * np.linalg.norm(v0)
    # with one value everywhere the uncentered statistic is m |v0|
    np.testing.assert_allclose(cu, cm * np.linalg.norm(v0), rtol=1e-12, atol=1e-300)


@pytest.mark.parametrize("seed", range(4))
def test_uncentered_dominates_centered(seed):
    # Cauchy-Schwarz: |sum a v|^2 <= (sum a) (sum a |v|^2)
    rng = np.random.default_rng(10 + seed)
    n, d = 150, 32
    s, perm = _rank(rng, n)
    v = rng.standard_t(3, size=(n, d))
    cc, _ = oracle.curves(s, perm, v, "centered")
    cu, _ = oracle.curves(s, perm, v, "uncentered")
    assert np.all(cu >= cc * (1 - 1e-12))


def test_uniform_allocator_splits_the_real_budget_evenly():
    rng = np.random.default_rng(3)
    H, n, n_keep = 8, 500, 51
    c32 = np.sort(rng.random((H, n)).astype(np.float32), axis=1)[:, ::-1].copy()
    b, rep = oracle.allocate(c32, n_keep, allocator="uniform")
    assert rep == 0 and list(b) == [n_keep - 1] * H
    b, _ = oracle.allocate(c32, n_keep, allocator="uniform", slot=False)
    assert list(b) == [n_keep] * H


def _convex_curves(rng, H, n):
    # decreasing convex curves: nonnegative decreasing marginals, summed from the right
    out = np.zeros((H, n), np.float32)
    for h in range(H):
        dec = np.sort(rng.random(n - 1) * rng.uniform(0.2, 3.0))[::-1]
        c = np.concatenate([np.cumsum(dec[::-1])[::-1], [0.0]])
        out[h] = c.astype(np.float32)
    return out


@pytest.mark.parametrize("seed", range(5))
def test_greedy_marginal_is_optimal_on_convex_curves(seed):
    # brute force over every budget vector with sum B_real and b_h >= b_min
    rng = np.random.default_rng(20 + seed)
    H, n, n_keep = 3, 9, 4
    c32 = _convex_curves(rng, H, n)
    B_real, b_min = oracle.budget_params(H, n, n_keep, 0.2)
    best = min(sum(float(c32[h, b[h]]) for h in range(H))
               for b in itertools.product(range(b_min, n), repeat=H) if sum(b) == B_real)
    b, _ = oracle.allocate(c32, n_keep, allocator="greedy")
    assert sum(b) == B_real and min(b) >= b_min
    assert abs(sum(float(c32[h, b[h]]) for h in range(H)) - best) <= 1e-6
    bl, _ = oracle.allocate(c32, n_keep)
    assert abs(sum(float(c32[h, bl[h]]) for h in range(H)) - best) <= 1e-6


def test_greedy_marginal_starts_every_head_at_b_min():
    rng = np.random.default_rng(4)
    H, n, n_keep = 4, 200, 20
    c32 = np.sort(rng.random((H, n)).astype(np.float32), axis=1)[:, ::-1].copy()
    B_real, b_min = oracle.budget_params(H, n, n_keep, 0.2)
    b, rep = oracle.allocate(c32, n_keep, allocator="greedy")
    assert sum(b) == B_real and rep == B_real - H * b_min


def test_no_slot_budget_algebra():
    # the slot's live row becomes one more real token per head
    assert oracle.budget_params(8, 100, 10, 0.2, slot=False) == (80, 2)
    assert oracle.budget_params(8, 100, 10, 0.2) == (72, 1)
    assert oracle.budget_params(4, 100, 99, 0.2, slot=False)[0] == 4 * 99
    with pytest.raises(oracle.OracleError):
        oracle.budget_params(4, 100, 100, 0.2, slot=False)   # a head keeps at most n - 1
    assert oracle.budget_params(4, 100, 1, 0.0, slot=False) == (4, 1)
    with pytest.raises(oracle.OracleError):
        oracle.budget_params(4, 100, 1, 0.0)                 # with the slot n_keep >= 2


@pytest.mark.parametrize("variant", [
    dict(statistic="tail_mass"), dict(statistic="uncentered"), dict(allocator="uniform"),
    dict(allocator="greedy"), dict(slot=False)])
def test_compress_block_variants_keep_the_budget_identities(variant):
    rng = np.random.default_rng(5)
    n, H, G, d, w, n_keep = 400, 4, 2, 16, 8, 41
    q = rng.normal(size=(w, H * G, d))
    k = rng.normal(size=(n, H, d))
    v = rng.standard_t(3, size=(n, H, d))
    out = oracle.compress_block(q, k, v, n_keep, d ** -0.5, **variant)
    slot = variant.get("slot", True)
    B_real, b_min = oracle.budget_params(H, n, n_keep, 0.2, slot=slot)
    assert int(out["budgets"].sum()) == B_real
    assert [len(x) for x in out["kept"]] == list(out["budgets"])
    for h in range(H):   # the curves follow the chosen statistic on the block's own order
        _, c32 = oracle.curves(out["s32"][h], out["perm"][h], v[:, h],
                               variant.get("statistic", "centered"))
        np.testing.assert_array_equal(out["c32"][h], c32)
    if variant.get("allocator") == "uniform":
        assert list(out["budgets"]) == [n_keep - 1] * H
