"""CPU pins of the oracle's decode over the packed cache and of the terms of
the future-query lift theorem (section "Scoped guarantees behind CertKV")."""
import math

import numpy as np
import pytest
import scipy.special

import oracle


def test_decode_known_logits_match_library_softmax():
    # keys along the first axis only, q = e_1 / scale: the logits are exactly t
    rng = np.random.default_rng(0)
    nk, d, scale = 37, 16, 0.5
    t = rng.normal(size=nk) * 3.0
    kp = np.zeros((nk, d))
    kp[:, 0] = t
    vp = rng.normal(size=(nk, d))
    q = np.zeros((2, d))
    q[:, 0] = 1.0 / scale
    out, lse = oracle.decode(q, kp, vp, scale)
    w = scipy.special.softmax(t)
    for r in range(2):
        np.testing.assert_allclose(out[r], w @ vp, rtol=1e-12, atol=1e-12)
        assert abs(lse[r] - scipy.special.logsumexp(t)) <= 1e-12


def test_decode_single_row_and_uniform_logits():
    rng = np.random.default_rng(1)
    kp = rng.normal(size=(1, 8))
    vp = rng.normal(size=(1, 8))
    q = rng.normal(size=(3, 8))
    out, lse = oracle.decode(q, kp, vp, 0.3)
    np.testing.assert_array_equal(out, np.repeat(vp, 3, axis=0))  # a weight of exactly 1
    np.testing.assert_allclose(lse, 0.3 * (q @ kp[0]), rtol=1e-13)
    kp5 = rng.normal(size=(5, 8))
    vp5 = rng.normal(size=(5, 8))
    out, lse = oracle.decode(np.zeros((2, 8)), kp5, vp5, 1.0)
    np.testing.assert_allclose(out, np.repeat(vp5.mean(axis=0, keepdims=True), 2, axis=0),
                               rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lse, math.log(5.0), rtol=1e-15)


def test_decode_is_invariant_to_row_order():
    rng = np.random.default_rng(2)
    kp = rng.normal(size=(64, 16))
    vp = rng.normal(size=(64, 16))
    q = rng.normal(size=(4, 16))
    perm = rng.permutation(64)
    o1, l1 = oracle.decode(q, kp, vp, 0.25)
    o2, l2 = oracle.decode(q, kp[perm], vp[perm], 0.25)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13)


def test_one_evicted_key_slot_reproduces_full_attention():
    # The slot of a one-key tail is that key itself: compressed attention is
    # exact attention, p = q and a = r.
    rng = np.random.default_rng(3)
    n, d, j = 50, 16, 17
    k = rng.normal(size=(n, d))
    v = rng.normal(size=(n, d))
    q = rng.normal(size=d)
    scale = 1.0 / math.sqrt(d)
    kept = np.ones(n, bool)
    kept[j] = False
    r = np.zeros(n)
    r[j] = 1.0
    t = oracle.lift_terms(q, k, v, kept, r, k[j], v[j], scale)
    assert t["err"] <= 1e-13 and abs(t["p"] - t["q"]) <= 1e-15 and t["l1"] <= 1e-12
    kp = np.concatenate([k[kept], k[j:j + 1]])
    vp = np.concatenate([v[kept], v[j:j + 1]])
    o_c, _ = oracle.decode(q[None], kp, vp, scale)
    o_f, _ = oracle.decode(q[None], k, v, scale)
    np.testing.assert_allclose(o_c, o_f, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("seed", range(6))
def test_lift_bound_and_sigmoid_identities(seed):
    rng = np.random.default_rng(100 + seed)
    n, d = 200, 32
    scale = 1.0 / math.sqrt(d)
    k = rng.normal(size=(n, d)) * (1.0 + seed)
    v = rng.normal(size=(n, d))
    s = rng.gamma(0.3, size=n)                      # heavy-tailed positive scores
    kept = np.zeros(n, bool)
    kept[np.argsort(-s, kind="stable")[: n // 3]] = True
    r = np.where(kept, 0.0, s)
    r /= r.sum()
    kslot, vslot = r @ k, r @ v                     # the slot's value is sum_T r_j v_j
    q = rng.normal(size=d) * 2.0
    t = oracle.lift_terms(q, k, v, kept, r, kslot, vslot, scale)
    bound = t["v_max"] * (2.0 * abs(t["p"] - t["q"]) + min(t["p"], t["q"]) * t["l1"])
    assert t["err"] <= bound * (1 + 1e-12) + 1e-15, (t, bound)
    assert abs(t["p"] - t["q"]) <= math.tanh(abs(t["lam_T"] - t["z_slot"]) / 4.0) + 1e-15
    # p = sigmoid(Lambda_T - log Z_S), q = sigmoid(z* - log Z_S), from this
    # test's own partitions
    z = scale * (k @ q)
    log_zs = scipy.special.logsumexp(z[kept])
    assert abs(t["lam_T"] - scipy.special.logsumexp(z[~kept])) <= 1e-12
    assert abs(t["z_slot"] - scale * float(kslot @ q)) <= 1e-12
    assert abs(t["p"] - scipy.special.expit(t["lam_T"] - log_zs)) <= 1e-12
    assert abs(t["q"] - scipy.special.expit(t["z_slot"] - log_zs)) <= 1e-12
    assert abs(t["v_max"] - np.linalg.norm(v, axis=1).max()) <= 1e-12
