"""Host-side checks of the C ABI: the library loads, exports every entry point
the header declares, and validates arguments (CERTKV_DRY_RUN: nothing is
launched, so these run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2608_21541_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "certkv.h")

FAKE = 1 << 20  # aligned non-null stand-in pointer (never dereferenced in dry runs)


def declared_entry_points():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(certkv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = _lib.lib()
    names = declared_entry_points()
    assert len(names) >= 12
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(_lib.EXPORTS)


def problem(L=2, seqlens=(1000, 700), H=4, G=2, d=128, w=16, dtype=_lib.CERTKV_BF16, flags=None):
    cu = [0]
    for n in seqlens:
        cu.append(cu[-1] + n)
    arr = (ctypes.c_int64 * len(cu))(*cu)
    fl = (_lib.CERTKV_CAUSAL | _lib.CERTKV_DRY_RUN) if flags is None else flags
    p = _lib.Problem(L, len(seqlens), H, G, d, w, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int64)),
                     dtype, dtype, 0.0, fl, None)
    p._keep = arr
    return p


def tensor(ptr=FAKE, sl=8 * 4 * 128 * 1700, st=4 * 128, sh=128):
    return _lib.Tensor(ptr, sl, st, sh)


def ws_for(p, stage):
    n = _lib.lib().certkv_workspace_size(ctypes.byref(p), stage)
    return (FAKE if n else None), n


def status_name(st):
    return _lib.lib().certkv_status_string(st).decode()


def test_status_strings():
    for st in [0, -1, -2, -3, -4, -5, -6, -99]:
        assert isinstance(status_name(st), str) and status_name(st)


def test_dry_run_score_validation():
    L = _lib.lib()
    p = problem()
    ws, n = ws_for(p, _lib.STAGE_SCORE)
    assert n > 0

    def call(pp, q=None, k=None, nbytes=n, lse_in=None, lse_out=None):
        return L.certkv_score(ctypes.byref(pp), q or tensor(), k or tensor(), lse_in, FAKE, None,
                              lse_out, ws, nbytes, None)

    assert call(p) == _lib.CERTKV_OK
    assert call(p, nbytes=n - 256) == _lib.CERTKV_EWORKSPACE
    assert call(p, q=tensor(ptr=FAKE + 4)) == _lib.CERTKV_EINVAL
    assert call(p, q=tensor(st=4 * 128 + 4)) == _lib.CERTKV_EINVAL
    assert call(problem(d=96)) == _lib.CERTKV_EUNSUPPORTED
    assert call(problem(w=701)) == _lib.CERTKV_EINVAL
    assert call(problem(H=65)) == _lib.CERTKV_EUNSUPPORTED
    assert call(problem(w=64, G=9)) == _lib.CERTKV_EUNSUPPORTED  # 576 window rows > 512
    assert call(problem(flags=_lib.CERTKV_DRY_RUN | 256)) == _lib.CERTKV_EINVAL
    # one statistic and one allocator at a time
    both_stats = _lib.CERTKV_STAT_UNCENTERED | _lib.CERTKV_STAT_TAIL_MASS
    both_allocs = _lib.CERTKV_ALLOC_UNIFORM | _lib.CERTKV_ALLOC_GREEDY
    assert call(problem(flags=_lib.CERTKV_DRY_RUN | both_stats)) == _lib.CERTKV_EINVAL
    assert call(problem(flags=_lib.CERTKV_DRY_RUN | both_allocs)) == _lib.CERTKV_EINVAL
    for f in (_lib.CERTKV_STAT_UNCENTERED, _lib.CERTKV_STAT_TAIL_MASS, _lib.CERTKV_ALLOC_UNIFORM,
              _lib.CERTKV_ALLOC_GREEDY, _lib.CERTKV_NO_SLOT):
        assert call(problem(flags=_lib.CERTKV_DRY_RUN | _lib.CERTKV_CAUSAL | f)) == _lib.CERTKV_OK
    # the caller's row log-sum-exp and the row log-sum-exp output are plain
    # optional device pointers
    assert call(p, lse_in=FAKE, lse_out=FAKE) == _lib.CERTKV_OK
    assert L.certkv_score(ctypes.byref(p), tensor(), tensor(), None, None, None, None, ws, n,
                          None) == _lib.CERTKV_EINVAL  # scores are required


def test_dry_run_allocate_budget_checks():
    L = _lib.lib()
    p = problem()
    ws, n = ws_for(p, _lib.STAGE_ALLOCATE)

    def call(nk, alpha=0.2, steps=40):
        arr = (ctypes.c_int32 * 2)(*nk)
        return L.certkv_allocate(ctypes.byref(p), FAKE, tensor(), arr, alpha, steps, FAKE, None,
                                 None, None, ws, n, None)

    assert call([101, 71]) == _lib.CERTKV_OK
    assert call([1, 71]) == _lib.CERTKV_EINFEASIBLE       # n_keep >= 2
    assert call([1001, 71]) == _lib.CERTKV_EINFEASIBLE    # n_keep <= n
    assert call([700, 700]) == _lib.CERTKV_OK             # keep all of sequence 2
    assert call([101, 71], alpha=1.5) == _lib.CERTKV_EINVAL
    assert call([101, 71], steps=-1) == _lib.CERTKV_EINVAL
    assert L.certkv_allocate(ctypes.byref(p), FAKE, tensor(), None, 0.2, 40, FAKE, None, None,
                             None, ws, n, None) == _lib.CERTKV_EINVAL


def test_dry_run_compress_and_select():
    L = _lib.lib()
    p = problem()
    ws, n = ws_for(p, _lib.STAGE_COMPRESS)
    out = _lib.Outputs(*([FAKE] * 11 + [None, None, None, None, None]))
    nk = (ctypes.c_int32 * 2)(101, 71)
    assert L.certkv_compress(ctypes.byref(p), tensor(), tensor(), tensor(), None, nk, 0.2, 40,
                             ctypes.byref(out), ws, n, None) == _lib.CERTKV_OK
    out.kept_mask = FAKE + 8  # the kept mask must be 16-byte aligned
    assert L.certkv_compress(ctypes.byref(p), tensor(), tensor(), tensor(), FAKE, nk, 0.2, 40,
                             ctypes.byref(out), ws, n, None) == _lib.CERTKV_EINVAL
    out.kept_mask = FAKE
    out.lse = FAKE
    assert L.certkv_compress(ctypes.byref(p), tensor(), tensor(), tensor(), FAKE, nk, 0.2, 40,
                             ctypes.byref(out), ws, n, None) == _lib.CERTKV_OK
    out.kept_idx = None
    assert L.certkv_compress(ctypes.byref(p), tensor(), tensor(), tensor(), None, nk, 0.2, 40,
                             ctypes.byref(out), ws, n, None) == _lib.CERTKV_EINVAL
    ws2, n2 = ws_for(p, _lib.STAGE_SELECT)
    assert L.certkv_select(ctypes.byref(p), FAKE, FAKE, 5, 0.9, FAKE, FAKE, 10, None, ws2, n2,
                           None) == _lib.CERTKV_EINVAL  # bad mode
    assert L.certkv_select(ctypes.byref(p), FAKE, FAKE, _lib.CERTKV_SELECT_COVERAGE, 1.5, FAKE,
                           FAKE, 1 << 30, None, ws2, n2, None) == _lib.CERTKV_EINVAL
    assert L.certkv_select(ctypes.byref(p), FAKE, FAKE, _lib.CERTKV_SELECT_COVERAGE, 0.9, FAKE,
                           FAKE, 1 << 30, None, ws2, n2, None) == _lib.CERTKV_OK
    assert L.certkv_select(ctypes.byref(p), FAKE, FAKE, _lib.CERTKV_SELECT_BUDGET, 0.9, FAKE,
                           FAKE, 10, FAKE, ws2, n2, None) == _lib.CERTKV_OK
    assert L.certkv_select(ctypes.byref(p), FAKE, FAKE, _lib.CERTKV_SELECT_BUDGET, 0.9, FAKE,
                           FAKE, 10, FAKE + 4, ws2, n2, None) == _lib.CERTKV_EINVAL


def test_keep_window_needs_room_for_the_window():
    L = _lib.lib()
    p = problem(flags=_lib.CERTKV_CAUSAL | _lib.CERTKV_DRY_RUN | _lib.CERTKV_KEEP_WINDOW)
    ws, n = ws_for(p, _lib.STAGE_ALLOCATE)

    def call(nk):
        arr = (ctypes.c_int32 * 2)(*nk)
        return L.certkv_allocate(ctypes.byref(p), FAKE, tensor(), arr, 0.2, 40, FAKE, None,
                                 None, None, ws, n, None)

    # H = 4, w = 16: b_min = floor(0.2 * (4 n_keep - 4) / 4) must reach 16
    assert call([101, 81]) == _lib.CERTKV_OK          # b_min = 20, 16
    assert call([101, 71]) == _lib.CERTKV_EINFEASIBLE  # b_min = 14 < 16 for sequence 2


def test_fp32_values_need_head_dim_64():
    L = _lib.lib()
    p = problem(dtype=_lib.CERTKV_F32, d=128, w=8, G=1)
    ws, n = ws_for(p, _lib.STAGE_ALLOCATE)
    nk = (ctypes.c_int32 * 2)(101, 71)
    assert L.certkv_allocate(ctypes.byref(p), FAKE, tensor(), nk, 0.2, 40, FAKE, None, None, None,
                             ws, n, None) == _lib.CERTKV_EUNSUPPORTED
    p64 = problem(dtype=_lib.CERTKV_F32, d=64, w=8, G=1)
    ws, n = ws_for(p64, _lib.STAGE_ALLOCATE)
    assert L.certkv_allocate(ctypes.byref(p64), FAKE, tensor(sl=0, st=256, sh=64), nk, 0.2, 40,
                             FAKE, None, None, None, ws, n, None) == _lib.CERTKV_OK


def test_workspace_size_zero_on_invalid():
    L = _lib.lib()
    assert L.certkv_workspace_size(ctypes.byref(problem(d=96)), _lib.STAGE_COMPRESS) == 0
    assert L.certkv_workspace_size(ctypes.byref(problem()), 99) == 0


def test_profile_api_without_launches():
    L = _lib.lib()
    assert L.certkv_profile_enable(1) == 0
    names = (ctypes.c_char * 64 * 8)()
    assert L.certkv_profile_read(names, None, None, 8) == 0
    L.certkv_profile_reset()
    assert L.certkv_profile_enable(0) == 0


def test_dry_run_decode_validation():
    L = _lib.lib()
    p = problem()
    n = L.certkv_decode_workspace_size(ctypes.byref(p), 8, 0)
    assert n > 0
    # the partials grow with the number of new queries and never shrink; a
    # segment bound below the longest sequence shrinks them
    assert L.certkv_decode_workspace_size(ctypes.byref(p), 64, 0) >= n
    plong = problem(seqlens=(5000, 700))
    assert 0 < L.certkv_decode_workspace_size(ctypes.byref(plong), 8, 100) < \
        L.certkv_decode_workspace_size(ctypes.byref(plong), 8, 0)
    assert L.certkv_decode_workspace_size(ctypes.byref(p), 0, 0) == 0
    assert L.certkv_decode_workspace_size(ctypes.byref(p), 8, -1) == 0

    def call(pp=p, tq=8, q=None, kp=FAKE, vp=FAKE, off=FAKE, out=FAKE, ws=FAKE, nbytes=n, mr=0):
        q = tensor() if q is None else q
        return L.certkv_decode(ctypes.byref(pp), q, tq, mr, kp, vp, off, out, None, ws, nbytes,
                               None)

    assert call() == _lib.CERTKV_OK
    assert call(tq=0) == _lib.CERTKV_EINVAL
    assert call(tq=257) == _lib.CERTKV_EUNSUPPORTED          # tq * G = 514 rows > 512
    assert call(q=tensor(ptr=FAKE + 2)) == _lib.CERTKV_EINVAL
    assert call(q=tensor(st=4 * 128 + 4)) == _lib.CERTKV_EINVAL
    assert call(kp=FAKE + 8) == _lib.CERTKV_EINVAL
    assert call(off=None) == _lib.CERTKV_EINVAL
    assert call(out=None) == _lib.CERTKV_EINVAL
    assert call(ws=None) == _lib.CERTKV_EWORKSPACE
    assert call(nbytes=n - 1) == _lib.CERTKV_EWORKSPACE
    assert call(ws=FAKE + 64) == _lib.CERTKV_EINVAL
    assert call(mr=-1) == _lib.CERTKV_EINVAL
    assert call(mr=100, nbytes=L.certkv_decode_workspace_size(ctypes.byref(p), 8, 100)) == \
        _lib.CERTKV_OK
    pf = problem(dtype=_lib.CERTKV_F32)
    nf = L.certkv_decode_workspace_size(ctypes.byref(pf), 8, 0)
    assert call(pp=pf, nbytes=nf) == _lib.CERTKV_EUNSUPPORTED


def test_dry_run_cluster_validation():
    L = _lib.lib()
    no_slot = _lib.CERTKV_CAUSAL | _lib.CERTKV_DRY_RUN | _lib.CERTKV_NO_SLOT
    p = problem(flags=no_slot)
    p_slot = problem()
    t = tensor()

    def tail(m=8, perm=FAKE, bud=FAKE, out=FAKE, pp=p):
        return L.certkv_cluster_tail(ctypes.byref(pp), t, t, perm, bud, m, out, out, out, out,
                                     out, out, None)
    assert tail() == _lib.CERTKV_OK
    assert tail(m=0) == _lib.CERTKV_EINVAL and tail(m=65) == _lib.CERTKV_EINVAL
    assert tail(perm=None) == _lib.CERTKV_EINVAL and tail(out=None) == _lib.CERTKV_EINVAL
    # the summaries replace the slot: a problem with the slot is rejected
    assert tail(pp=p_slot) == _lib.CERTKV_EINVAL
    n = L.certkv_decode_workspace_size(ctypes.byref(p), 8, 0)

    def dec(m=8, cl=FAKE, pp=p):
        return L.certkv_decode_clustered(ctypes.byref(pp), tensor(), 8, 0, FAKE, FAKE, FAKE, m,
                                         cl, cl, cl, cl, cl, cl, FAKE, None, None, FAKE, n, None)
    assert dec() == _lib.CERTKV_OK
    assert dec(m=0) == _lib.CERTKV_EINVAL and dec(cl=None) == _lib.CERTKV_EINVAL
    # segments that end in a slot row would count the evicted mass twice
    assert dec(pp=p_slot) == _lib.CERTKV_EINVAL
    # the plain decode takes either kind of segment
    assert L.certkv_decode(ctypes.byref(p_slot), tensor(), 8, 0, FAKE, FAKE, FAKE, FAKE, None,
                           FAKE, n, None) == _lib.CERTKV_OK
