"""CPU pins of the oracle's clustered tail summaries and their runtime
certificate (appendix, deterministic output-error bound for clustered tail
summaries)."""
import math

import numpy as np
import pytest

import oracle


def _head(rng, n, d, b):
    # fp32-representable inputs: a one-key mean is then stored exactly
    k = rng.normal(size=(n, d)).astype(np.float32).astype(np.float64)
    v = rng.normal(size=(n, d)).astype(np.float32).astype(np.float64)
    s = rng.gamma(0.4, size=n).astype(np.float32)
    perm = oracle.order(s)
    return k, v, perm


def test_singleton_clusters_reproduce_exact_attention_with_zero_bound():
    rng = np.random.default_rng(0)
    n, d, b = 60, 16, 20
    k, v, perm = _head(rng, n, d, b)
    cl = oracle.cluster_summaries(perm, b, k, v, n - b, bf16=False)
    assert (cl["count"] == 1).all() and (cl["R"] == 0).all() and (cl["rho"] == 0).all()
    kept = perm[:b]
    q = rng.normal(size=d)
    scale = 1 / math.sqrt(d)
    out, c = oracle.cluster_estimate(q, k[kept], v[kept], cl, scale)
    ref, lse = oracle.decode(q[None], k, v, scale)
    np.testing.assert_allclose(out, ref[0], rtol=1e-12, atol=1e-14)
    assert abs(c["lse"] - lse[0]) <= 1e-12
    assert c["bound"] == 0.0 and c["dz"] == 0.0 and c["dn"] == 0.0


def test_identical_evicted_rows_give_an_exact_single_cluster():
    rng = np.random.default_rng(1)
    n, d, b = 50, 8, 10
    k, v, perm = _head(rng, n, d, b)
    ev = perm[b:]
    k[ev] = rng.normal(size=d)
    v[ev] = rng.normal(size=d)
    cl = oracle.cluster_summaries(perm, b, k, v, 1, bf16=False)
    assert cl["count"][0] == n - b and cl["R"][0] <= 1e-6 and cl["rho"][0] <= 1e-6
    q = rng.normal(size=d)
    out, c = oracle.cluster_estimate(q, k[perm[:b]], v[perm[:b]], cl, 0.3)
    ref, _ = oracle.decode(q[None], k, v, 0.3)
    np.testing.assert_allclose(out, ref[0], rtol=1e-6, atol=1e-9)


def test_counts_cover_the_evicted_ranks():
    rng = np.random.default_rng(2)
    n, d, b = 1003, 8, 100
    k, v, perm = _head(rng, n, d, b)
    for m in (1, 7, 64, 1000):
        cl = oracle.cluster_summaries(perm, b, k, v, m)
        assert int(cl["count"].sum()) == n - b
        assert cl["count"].max() == -(-(n - b) // m)
    assert oracle.cluster_summaries(perm, b, k, v, 4)["vmax_kept"] >= \
        np.linalg.norm(v[perm[:b]], axis=1).max() * (1 - 1e-7)


@pytest.mark.parametrize("seed", range(8))
def test_certificate_bounds_the_true_error(seed):
    # the evicted ranks form m tight key clusters (one centre per contiguous
    # group), so the logit radii are small, the condition D_Z <= Zhat / 3 holds
    # and the bound is checked against the exact error; the structural form
    # dominates the bound
    rng = np.random.default_rng(50 + seed)
    n, d, b, m = 400, 16, 40, 8
    s = rng.gamma(0.4, size=n).astype(np.float32)
    perm = oracle.order(s)
    k = rng.normal(size=(n, d))
    v = rng.normal(size=(n, d))
    centres = rng.normal(size=(m, d))
    ev = perm[b:]
    grp = np.arange(n - b) // ((n - b) // m)
    k[ev] = centres[grp] + 0.02 * rng.normal(size=(n - b, d))
    cl = oracle.cluster_summaries(perm, b, k, v, m)
    scale = 1 / math.sqrt(d)
    finite = 0
    for _ in range(6):
        q = rng.normal(size=d)
        out, c = oracle.cluster_estimate(q, k[perm[:b]], v[perm[:b]], cl, scale)
        ref, _ = oracle.decode(q[None], k, v, scale)
        err = float(np.linalg.norm(out - ref[0]))
        if math.isfinite(c["bound"]):
            finite += 1
            assert err <= c["bound"] * (1 + 1e-9), (err, c)
            assert c["bound"] <= c["structural"] * (1 + 1e-9)
        else:
            assert c["dz"] > 1 / 3
    assert finite >= 4   # the certificate is not vacuous here


def test_radii_hand_computed_sampled_centre():
    # One group of 192 members in rank order: member stride S = 192 / 64 = 3,
    # so the sample is ranks 0, 3, 6, ...  The keys of sampled ranks are
    # (0, 0), the others (6, 0); the values of sampled ranks are (0, 3), the
    # others (0, -3).  With fp32 storage: c_k = (0, 0), kbar = (4, 0);
    # c_v = (0, 3), vbar = (0, -1).  Then
    #   R   = max |k - c_k| + |c_k - kbar| = 6 + 4 = 10   (exact max: 4)
    #   rho = max |v - c_v| + |c_v - vbar| = 6 + 4 = 10   (exact max: 4)
    n = 192
    samp = np.arange(n) % 3 == 0
    k = np.where(samp[:, None], [[0.0, 0.0]], [[6.0, 0.0]])
    v = np.where(samp[:, None], [[0.0, 3.0]], [[0.0, -3.0]])
    perm = np.arange(n, dtype=np.int32)
    cl = oracle.cluster_summaries(perm, 0, k, v, 1, bf16=False)
    np.testing.assert_array_equal(cl["kbar"][0], [4.0, 0.0])
    np.testing.assert_array_equal(cl["vbar"][0], [0.0, -1.0])
    assert cl["R"][0] == 10.0 and cl["rho"][0] == 10.0
    # groups of at most 64 members use them all (S = 1): c is the exact mean
    # and the radii are the exact maxima up to the storage rounding
    k = np.array([[0.0, 0.0], [2.0, 0.0], [4.0, 0.0]])
    cl = oracle.cluster_summaries(np.arange(3, dtype=np.int32), 0, k, k, 1, bf16=False)
    assert cl["R"][0] == 2.0
    # 2000 members: S = 2000 / 64 = 31 clamped to 16, sample ranks 0, 16, ...
    rng = np.random.default_rng(5)
    k = rng.integers(-8, 9, size=(2000, 4)).astype(np.float64)
    v = rng.integers(-8, 9, size=(2000, 4)).astype(np.float64)
    perm = rng.permutation(2000).astype(np.int32)
    cl = oracle.cluster_summaries(perm, 0, k, v, 1, bf16=False)
    for x, bar, r in ((k, cl["kbar"][0], cl["R"][0]), (v, cl["vbar"][0], cl["rho"][0])):
        c = x[perm[::16]].mean(0)
        want = np.linalg.norm(x - c, axis=1).max() + np.linalg.norm(c - bar)
        assert want <= r <= want * (1 + 2 ** -22)


@pytest.mark.parametrize("bf16", [False, True])
def test_radii_bound_every_member_and_stay_tight(bf16):
    # the cluster-radii equation: every member within R of the stored key
    # representative and within rho of the stored value one; on Gaussian
    # groups of ~1000 members the sampled centre is close to the mean, so the
    # radii exceed the exact maxima by a few percent only
    rng = np.random.default_rng(6)
    n, d, b = 4200, 32, 200
    k, v, perm = _head(rng, n, d, b)
    m = 4
    cl = oracle.cluster_summaries(perm, b, k, v, m, bf16=bf16)
    E = perm[b:]
    cs = -(-len(E) // m)
    for g in range(m):
        mem = E[g * cs:(g + 1) * cs]
        ek = np.linalg.norm(k[mem] - cl["kbar"][g], axis=1).max()
        ev = np.linalg.norm(v[mem] - cl["vbar"][g], axis=1).max()
        assert ek <= cl["R"][g] <= 1.15 * ek
        assert ev <= cl["rho"][g] <= 1.15 * ev
