"""TEST INFRASTRUCTURE: ctypes front end of the fp64 CPU oracle.

The oracle (certkv_oracle.c) is a plain, slow implementation of the CertKV
compression pass written from the paper ("Beyond Sparse Weights: When Is
Attention Compressible?", Section 4.1 and the appendix's Algorithm 1).  Only
tests/, the smoke check and the benchmark's cpu_baseline leg may import this
package.  It shares no code with the HIP product path and never imports it.

Every wrapper takes numpy arrays; inputs are converted to contiguous float64
(bf16 and fp32 values convert exactly).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_dbl = ctypes.c_double
_p = ctypes.c_void_p

ORA_OK = 0
ORA_EINVAL = -1
ORA_EINFEASIBLE = -3
ORA_ENONFINITE = -4


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"oracle {what} failed with status {code}")
        self.code = code


def lib():
    """Load (building first if absent) libcertkv_oracle.so."""
    global _LIB
    if _LIB is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        L.ora_scores.argtypes = [_i64, _i32, _i32, _p, _p, _p, _dbl, _i32, _p, _p]
        L.ora_order.argtypes = [_i64, _p, _p]
        L.ora_order_window.argtypes = [_i64, _p, _i64, _p]
        L.ora_normalize.argtypes = [_i64, _p, _p]
        L.ora_curves.argtypes = [_i64, _i32, _p, _p, _p, _p, _p]
        L.ora_budget_params.argtypes = [_i32, _i64, _i64, _dbl, _p, _p]
        L.ora_argmin_penalized.argtypes = [_p, _i64, _i64, _dbl]
        L.ora_argmin_penalized.restype = _i64
        L.ora_allocate.argtypes = [_i32, _i64, _p, _i64, _dbl, _i32, _p, _p, _p]
        L.ora_select.argtypes = [_i64, _p, _i64, _p]
        L.ora_coverage.argtypes = [_i64, _p, _p, _dbl, _i64, _p]
        L.ora_tail.argtypes = [_i64, _i32, _p, _p, _i64, _p, _p, _p, _p, _p]
        L.ora_decode.argtypes = [_i64, _i32, _i32, _p, _p, _p, _dbl, _p, _p]
        L.ora_lift_terms.argtypes = [_i64, _i32, _p, _p, _p, _p, _p, _p, _p, _dbl, _p]
        L.ora_f32_to_bf16.argtypes = [ctypes.c_float]
        L.ora_f32_to_bf16.restype = ctypes.c_uint16
        L.ora_row_error.argtypes = [_i64, _i32, _p, _p, _p, _p]
        L.ora_row_error.restype = _dbl
        L.ora_compress_block.argtypes = [
            _i64, _i32, _i32, _i32, _i32, _p, _p, _p, _dbl, _i32, _i64, _dbl,
            _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p]
        L.ora_curves_stat.argtypes = [_i64, _i32, _p, _p, _p, _i32, _p, _p]
        L.ora_budget_params_slot.argtypes = [_i32, _i64, _i64, _dbl, _i32, _p, _p]
        L.ora_allocate_variant.argtypes = [_i32, _i64, _p, _i64, _dbl, _i32, _i32, _i32, _p,
                                           _p, _p]
        L.ora_compress_block_variant.argtypes = [
            _i64, _i32, _i32, _i32, _i32, _p, _p, _p, _dbl, _i32, _i64, _dbl,
            _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p]
        L.ora_cluster_summaries.argtypes = [_i64, _i32, _p, _i64, _p, _p, _i32, _i32, _p, _p,
                                            _p, _p, _p, _p]
        L.ora_cluster_estimate.argtypes = [_i64, _i32, _p, _p, _p, _i32, _p, _p, _p, _p, _p,
                                           ctypes.c_float, _dbl, _p, _p]
        L.ora_num_threads.restype = ctypes.c_int
        _LIB = L
    return _LIB


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _f32(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float32))


def _i32a(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _ptr(a):
    return a.ctypes.data_as(_p) if a is not None else None


def _check(code, what):
    if code != ORA_OK:
        raise OracleError(code, what)


def num_threads():
    return lib().ora_num_threads()


def scores(q, qpos, k, scale, causal=True, with_lse=False):
    """Window-mass scores of one KV head.  q [M][d], qpos [M], k [n][d]."""
    q, k = _f64(q), _f64(k)
    qpos = np.ascontiguousarray(np.asarray(qpos, dtype=np.int64))
    M, d = q.shape
    n = k.shape[0]
    s = np.zeros(n, np.float64)
    lse = np.zeros(M, np.float64) if with_lse else None
    _check(lib().ora_scores(n, d, M, _ptr(q), _ptr(qpos), _ptr(k), float(scale),
                            int(bool(causal)), _ptr(s), _ptr(lse)), "scores")
    return (s, lse) if with_lse else s


def order(s32, keep_window=0):
    """Rank order (score descending, ties by position); keep_window = w puts the
    last w positions first, in ascending position."""
    s32 = _f32(s32)
    perm = np.zeros(s32.shape[0], np.int32)
    if keep_window:
        _check(lib().ora_order_window(s32.shape[0], _ptr(s32), int(keep_window), _ptr(perm)),
               "order_window")
    else:
        _check(lib().ora_order(s32.shape[0], _ptr(s32), _ptr(perm)), "order")
    return perm


def normalize(s32):
    s32 = _f32(s32)
    a = np.zeros(s32.shape[0], np.float64)
    _check(lib().ora_normalize(s32.shape[0], _ptr(s32), _ptr(a)), "normalize")
    return a


STATISTICS = {"centered": 0, "uncentered": 1, "tail_mass": 2}
ALLOCATORS = ("lagrangian", "uniform", "greedy")


def curves(s32, perm, v, statistic="centered"):
    """Returns (c fp64, c32 fp32) over b = 0..n-1; statistic is the centered
    dispersion (default), the uncentered one or the tail mass."""
    s32, perm, v = _f32(s32), _i32a(perm), _f64(v)
    n, d = v.shape
    c = np.zeros(n, np.float64)
    c32 = np.zeros(n, np.float32)
    if statistic == "centered":
        st = lib().ora_curves(n, d, _ptr(s32), _ptr(perm), _ptr(v), _ptr(c), _ptr(c32))
    else:
        st = lib().ora_curves_stat(n, d, _ptr(s32), _ptr(perm), _ptr(v),
                                   STATISTICS[statistic], _ptr(c), _ptr(c32))
    _check(st, "curves")
    return c, c32


def budget_params(H, n, n_keep, alpha=0.2, slot=True):
    br = np.zeros(1, np.int64)
    bm = np.zeros(1, np.int64)
    if slot:
        st = lib().ora_budget_params(H, n, n_keep, float(alpha), _ptr(br), _ptr(bm))
    else:
        st = lib().ora_budget_params_slot(H, n, n_keep, float(alpha), 0, _ptr(br), _ptr(bm))
    _check(st, "budget_params")
    return int(br[0]), int(bm[0])


def argmin_penalized(c32, lo, hi, lam):
    c32 = _f32(c32)
    return int(lib().ora_argmin_penalized(_ptr(c32), lo, hi, float(lam)))


def allocate(c32, n_keep, alpha=0.2, steps=40, with_lambda=False, allocator="lagrangian",
             slot=True):
    """c32 [H][n] fp32 -> (budgets [H], repairs[, (lambda_lo, lambda_hi)]).
    allocator: "lagrangian" (bisection + repair), "uniform" (B_real / H each)
    or "greedy" (the repair from b_min, i.e. no bisection step); slot=False
    is the no-slot budget algebra."""
    c32 = _f32(c32)
    H, n = c32.shape
    b = np.zeros(H, np.int32)
    rep = np.zeros(1, np.int64)
    lam = np.zeros(2, np.float64)
    assert allocator in ALLOCATORS
    if allocator == "lagrangian" and slot:
        st = lib().ora_allocate(H, n, _ptr(c32), n_keep, float(alpha), steps, _ptr(b),
                                _ptr(rep), _ptr(lam))
    else:
        st = lib().ora_allocate_variant(H, n, _ptr(c32), n_keep, float(alpha),
                                        0 if allocator == "greedy" else steps, int(slot),
                                        int(allocator == "uniform"), _ptr(b), _ptr(rep),
                                        _ptr(lam))
    _check(st, "allocate")
    if with_lambda:
        return b, int(rep[0]), (float(lam[0]), float(lam[1]))
    return b, int(rep[0])


def select(perm, b):
    perm = _i32a(perm)
    kept = np.zeros(int(b), np.int32)
    _check(lib().ora_select(perm.shape[0], _ptr(perm), int(b), _ptr(kept)), "select")
    return kept


def coverage(s32, perm, retain, k_min=1):
    s32, perm = _f32(s32), _i32a(perm)
    k = np.zeros(1, np.int64)
    _check(lib().ora_coverage(s32.shape[0], _ptr(s32), _ptr(perm), float(retain), int(k_min),
                              _ptr(k)), "coverage")
    return int(k[0])


def tail(s32, kept, k, v):
    """Returns (k_star [d], v_star [d], m) by direct sums over evicted keys."""
    s32, kept, k, v = _f32(s32), _i32a(kept), _f64(k), _f64(v)
    n, d = k.shape
    ks = np.zeros(d, np.float64)
    vs = np.zeros(d, np.float64)
    m = np.zeros(1, np.float64)
    _check(lib().ora_tail(n, d, _ptr(s32), _ptr(kept), kept.shape[0], _ptr(k), _ptr(v),
                          _ptr(ks), _ptr(vs), _ptr(m)), "tail")
    return ks, vs, float(m[0])


def f32_to_bf16_bits(x):
    """Round-to-nearest-even bf16 bit patterns of an fp32 array."""
    x = _f32(x).ravel()
    L = lib()
    return np.array([L.ora_f32_to_bf16(float(t)) for t in x], np.uint16)


def row_error(A, V, kept_mask, u=None):
    """| sum_{kept} A_j V_j + u - sum_j A_j V_j |_2 for one realized row."""
    A, V = _f64(A), _f64(V)
    if V.ndim == 1:
        V = V[:, None]
    mask = np.ascontiguousarray(np.asarray(kept_mask, dtype=np.uint8))
    uu = _f64(u) if u is not None else None
    return float(lib().ora_row_error(A.shape[0], V.shape[1], _ptr(A), _ptr(V), _ptr(mask),
                                     _ptr(uu)))


def variant_bits(statistic="centered", allocator="lagrangian", slot=True):
    """The oracle's variant bit mask of a one-factor ablation."""
    assert statistic in STATISTICS and allocator in ALLOCATORS
    return ((1 if statistic == "uncentered" else 2 if statistic == "tail_mass" else 0)
            | (4 if allocator == "uniform" else 8 if allocator == "greedy" else 0)
            | (0 if slot else 16))


def compress_block(q, k, v, n_keep, scale, causal=True, alpha=0.2, steps=40, s32_in=None,
                   keep_window=False, statistic="centered", allocator="lagrangian", slot=True):
    """One (layer, sequence) block end to end.

    q [w][H*G][d], k/v [n][H][d] (any float dtype; converted to fp64 exactly).
    s32_in [H][n] optional fp32 scores that replace the scoring step.
    keep_window ranks the w window keys first, so every head keeps them.
    Returns a dict of every intermediate and output.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    w, HG, d = q.shape
    n, H, d2 = k.shape
    assert d == d2 and HG % H == 0
    G = HG // H
    s = np.zeros((H, n), np.float64)
    s32 = np.zeros((H, n), np.float32)
    perm = np.zeros((H, n), np.int32)
    c32 = np.zeros((H, n), np.float32)
    b = np.zeros(H, np.int32)
    kept = np.zeros(H * n, np.int32)
    kept_off = np.zeros(H + 1, np.int64)
    ks = np.zeros((H, d), np.float64)
    vs = np.zeros((H, d), np.float64)
    m = np.zeros(H, np.float64)
    rep = np.zeros(1, np.int64)
    sin = _f32(s32_in) if s32_in is not None else None
    var = variant_bits(statistic, allocator, slot)
    if var == 0:
        st = lib().ora_compress_block(
            n, H, G, d, w, _ptr(q), _ptr(k), _ptr(v), float(scale), int(bool(causal)),
            int(n_keep), float(alpha), int(steps), int(bool(keep_window)), _ptr(sin), _ptr(s),
            _ptr(s32), _ptr(perm),
            _ptr(c32), _ptr(b), _ptr(kept), _ptr(kept_off), _ptr(ks), _ptr(vs), _ptr(m),
            _ptr(rep))
    else:
        st = lib().ora_compress_block_variant(
            n, H, G, d, w, _ptr(q), _ptr(k), _ptr(v), float(scale), int(bool(causal)),
            int(n_keep), float(alpha), int(steps), int(bool(keep_window)), var, _ptr(sin),
            _ptr(s), _ptr(s32), _ptr(perm),
            _ptr(c32), _ptr(b), _ptr(kept), _ptr(kept_off), _ptr(ks), _ptr(vs), _ptr(m),
            _ptr(rep))
    _check(st, "compress_block")
    return dict(s=s, s32=s32, perm=perm, c32=c32, budgets=b,
                kept=[kept[kept_off[h]:kept_off[h + 1]].copy() for h in range(H)],
                k_star=ks, v_star=vs, tail_mass=m, repairs=int(rep[0]))


def decode(q, kp, vp, scale):
    """Attention of query rows q [m][d] over a packed segment (kept rows and
    the slot row, kp/vp [nk][d]) with the plain softmax of Section 4.1's
    live rows: returns (out [m][d], lse [m]) in fp64."""
    q = _f64(np.atleast_2d(q))
    kp, vp = _f64(kp), _f64(vp)
    m, d = q.shape
    out = np.zeros((m, d))
    lse = np.zeros(m)
    _check(lib().ora_decode(kp.shape[0], m, d, _ptr(q), _ptr(kp), _ptr(vp), float(scale),
                            _ptr(out), _ptr(lse)), "decode")
    return out, lse


def lift_terms(q, k, v, kept_mask, r, kslot, vslot, scale):
    """Terms of the future-query lift theorem for one query row q [d] over the
    original keys k, v [n][d] with retained set kept_mask and slot (kslot,
    vslot), the slot value being sum_T r_j v_j: a dict with p, q (slot
    weight), l1 = ||a - r||_1, lam_T, z_slot, v_max and err = ||O - Ohat||_2."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    kept = np.ascontiguousarray(kept_mask, dtype=np.uint8)
    r, kslot, vslot = _f64(r), _f64(kslot), _f64(vslot)
    n, d = k.shape
    out = np.zeros(7)
    _check(lib().ora_lift_terms(n, d, _ptr(q), _ptr(k), _ptr(v), _ptr(kept), _ptr(r),
                                _ptr(kslot), _ptr(vslot), float(scale), _ptr(out)), "lift_terms")
    return dict(zip(["p", "q", "l1", "lam_T", "z_slot", "v_max", "err"], out.tolist()))


def cluster_summaries(perm, b, k, v, m, bf16=True):
    """Clustered tail summaries of one head: the evicted ranks b..n-1 in the
    order perm cut into m contiguous groups.  Returns dict(kbar [m][d],
    vbar [m][d] (as stored), count [m], R [m], rho [m] fp32, vmax_kept)."""
    perm, k, v = _i32a(perm), _f64(k), _f64(v)
    n, d = k.shape
    kbar = np.zeros((m, d), np.float64)
    vbar = np.zeros((m, d), np.float64)
    cnt = np.zeros(m, np.int32)
    R = np.zeros(m, np.float32)
    rho = np.zeros(m, np.float32)
    vk = np.zeros(1, np.float32)
    _check(lib().ora_cluster_summaries(n, d, _ptr(perm), int(b), _ptr(k), _ptr(v), int(m),
                                       int(bool(bf16)), _ptr(kbar), _ptr(vbar), _ptr(cnt),
                                       _ptr(R), _ptr(rho), _ptr(vk)), "cluster_summaries")
    return dict(kbar=kbar, vbar=vbar, count=cnt, R=R, rho=rho, vmax_kept=float(vk[0]))


def cluster_estimate(q, kp, vp, cl, scale):
    """The clustered-summary estimator and certificate for one query q [d]
    over kept rows kp, vp [nk][d] and the summaries cl (cluster_summaries).
    Returns (out [d], dict(lse, dz, dn, vmax, bound, structural))."""
    q, kp, vp = _f64(q), _f64(kp), _f64(vp)
    d = q.shape[0]
    nk = kp.shape[0]
    m = cl["count"].shape[0]
    out = np.zeros(d, np.float64)
    cert = np.zeros(6, np.float64)
    kb, vb = _f64(cl["kbar"]), _f64(cl["vbar"])
    cnt, R, rho = _i32a(cl["count"]), _f32(cl["R"]), _f32(cl["rho"])
    _check(lib().ora_cluster_estimate(nk, d, _ptr(q), _ptr(kp), _ptr(vp), m, _ptr(kb),
                                      _ptr(vb), _ptr(cnt), _ptr(R), _ptr(rho),
                                      float(cl["vmax_kept"]), float(scale), _ptr(out),
                                      _ptr(cert)), "cluster_estimate")
    return out, dict(lse=cert[0], dz=cert[1], dn=cert[2], vmax=cert[3], bound=cert[4],
                     structural=cert[5])
