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
