"""Python binding of libcertkv.so with the C entry points' names.

Argument marshalling only: shapes and dtypes are read off torch tensors,
outputs and the workspace are allocated with torch on the tensors' device,
and every step of the pass runs in the library's HIP kernels on the current
torch stream.  Layouts follow include/certkv.h.
"""
import ctypes
import math
from dataclasses import dataclass, field
from typing import List, Optional

import torch

from . import _lib
from ._lib import CertKVError


@dataclass
class ProblemSpec:
    layers: int
    kv_heads: int
    group: int
    head_dim: int
    window: int
    seqlens: List[int]
    dtype: torch.dtype = torch.bfloat16
    softmax_scale: float = 0.0
    causal: bool = True
    dry_run: bool = False
    keep_window: bool = False   # window keys ranked first, never evicted
    # one-factor ablations: "centered" | "uncentered" | "tail_mass";
    # "lagrangian" | "uniform" | "greedy"; slot=False gives the slot's row to
    # one more real token per head
    statistic: str = "centered"
    allocator: str = "lagrangian"
    slot: bool = True
    status: Optional[torch.Tensor] = None  # device int32 [1]: CERTKV_ENONFINITE on non-finite input
    _cu: object = field(default=None, repr=False)

    @property
    def batch(self):
        return len(self.seqlens)

    @property
    def total_tokens(self):
        return int(sum(self.seqlens))

    @property
    def units(self):
        return self.layers * self.batch * self.kv_heads

    def cu_seqlens(self):
        cu = [0]
        for n in self.seqlens:
            cu.append(cu[-1] + int(n))
        return cu

    def c_problem(self):
        cu = self.cu_seqlens()
        self._cu = (ctypes.c_int64 * len(cu))(*cu)  # kept alive with the spec
        dt = _dtype_code(self.dtype)
        flags = (_lib.CERTKV_CAUSAL if self.causal else 0) | (
            _lib.CERTKV_DRY_RUN if self.dry_run else 0) | (
            _lib.CERTKV_KEEP_WINDOW if self.keep_window else 0) | {
            "centered": 0, "uncentered": _lib.CERTKV_STAT_UNCENTERED,
            "tail_mass": _lib.CERTKV_STAT_TAIL_MASS}[self.statistic] | {
            "lagrangian": 0, "uniform": _lib.CERTKV_ALLOC_UNIFORM,
            "greedy": _lib.CERTKV_ALLOC_GREEDY}[self.allocator] | (
            0 if self.slot else _lib.CERTKV_NO_SLOT)
        st = self.status.data_ptr() if self.status is not None else None
        return _lib.Problem(self.layers, self.batch, self.kv_heads, self.group, self.head_dim,
                            self.window, ctypes.cast(self._cu, ctypes.POINTER(ctypes.c_int64)),
                            dt, dt, float(self.softmax_scale), flags, st)


def _dtype_code(dt):
    if dt == torch.bfloat16:
        return _lib.CERTKV_BF16
    if dt == torch.float32:
        return _lib.CERTKV_F32
    raise ValueError(f"unsupported dtype {dt}")


def _tensor(t: torch.Tensor) -> _lib.Tensor:
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("expected a [layers][tokens][heads][head_dim] tensor with contiguous last dim")
    return _lib.Tensor(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(st, what):
    if st != _lib.CERTKV_OK:
        raise CertKVError(st, what)


def workspace_size(spec: ProblemSpec, stage: int) -> int:
    p = spec.c_problem()
    return int(_lib.lib().certkv_workspace_size(ctypes.byref(p), stage))


def _workspace(spec, stage, device):
    n = workspace_size(spec, stage)
    if n == 0:
        return None, 0
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws, n


def _lse_shape(spec):
    return (spec.layers, spec.batch * spec.window, spec.kv_heads * spec.group)


def score(spec: ProblemSpec, q_win, k, with_ksum=False, lse_in=None, with_lse=False):
    """Window-mass scores [L][H][T] fp32; with_ksum adds sum_j (s_j)_+ k_j [U][d] fp64 and
    with_lse the row log-sum-exp [L][B*w][Hq] fp32 (in that order).  lse_in: the caller's
    row log-sum-exp in the same layout (the row-sum pass is then skipped)."""
    L = _lib.lib()
    dev = k.device
    scores = torch.empty((spec.layers, spec.kv_heads, spec.total_tokens), dtype=torch.float32,
                         device=dev)
    ksum = torch.empty((spec.units, spec.head_dim), dtype=torch.float64, device=dev) \
        if with_ksum else None
    lse = torch.empty(_lse_shape(spec), dtype=torch.float32, device=dev) if with_lse else None
    if lse_in is not None:
        assert lse_in.dtype == torch.float32 and lse_in.is_contiguous()
        assert tuple(lse_in.shape) == _lse_shape(spec)
    ws, n = _workspace(spec, _lib.STAGE_SCORE, dev)
    p = spec.c_problem()
    _check(L.certkv_score(ctypes.byref(p), _tensor(q_win), _tensor(k), _ptr(lse_in), _ptr(scores),
                          _ptr(ksum), _ptr(lse), _ptr(ws), n, _stream(dev)), "certkv_score")
    out = [scores] + ([ksum] if with_ksum else []) + ([lse] if with_lse else [])
    return out[0] if len(out) == 1 else tuple(out)


def score_noalloc(spec: ProblemSpec, q_win, k, scores, ksum=None, lse_out=None, lse_in=None):
    """certkv_score with the library's fixed device workspace: the caller
    passes every output (scores [L][H][T] fp32; optional ksum [U][d] fp64 and
    lse_out [L][B*w][Hq] fp32) and nothing is allocated."""
    L = _lib.lib()
    dev = k.device
    assert scores.dtype == torch.float32 and scores.is_contiguous()
    assert tuple(scores.shape) == (spec.layers, spec.kv_heads, spec.total_tokens)
    if ksum is not None:
        assert ksum.dtype == torch.float64 and tuple(ksum.shape) == (spec.units, spec.head_dim)
    for t in (lse_in, lse_out):
        if t is not None:
            assert t.dtype == torch.float32 and t.is_contiguous()
            assert tuple(t.shape) == _lse_shape(spec)
    p = spec.c_problem()
    _check(L.certkv_score_noalloc(ctypes.byref(p), _tensor(q_win), _tensor(k), _ptr(lse_in),
                                  _ptr(scores), _ptr(ksum), _ptr(lse_out), _stream(dev)),
           "certkv_score_noalloc")
    return scores


def allocate(spec: ProblemSpec, scores, v, n_keep, alpha=0.2, steps=40, with_perm=False,
             with_curves=False, with_vsum=False):
    """Budgets [U] int32 (+ perm, curves [L][H][T], vsum [U][d])."""
    L = _lib.lib()
    dev = v.device
    budgets = torch.empty(spec.units, dtype=torch.int32, device=dev)
    shape = (spec.layers, spec.kv_heads, spec.total_tokens)
    perm = torch.empty(shape, dtype=torch.int32, device=dev) if with_perm else None
    curves = torch.empty(shape, dtype=torch.float32, device=dev) if with_curves else None
    vsum = torch.empty((spec.units, spec.head_dim), dtype=torch.float64, device=dev) \
        if with_vsum else None
    nk = (ctypes.c_int32 * spec.batch)(*[int(x) for x in n_keep])
    ws, n = _workspace(spec, _lib.STAGE_ALLOCATE, dev)
    p = spec.c_problem()
    _check(L.certkv_allocate(ctypes.byref(p), _ptr(scores), _tensor(v), nk, float(alpha),
                             int(steps), _ptr(budgets), _ptr(perm), _ptr(curves), _ptr(vsum),
                             _ptr(ws), n, _stream(dev)), "certkv_allocate")
    out = {"budgets": budgets}
    if with_perm:
        out["perm"] = perm
    if with_curves:
        out["curves"] = curves
    if with_vsum:
        out["vsum"] = vsum
    return out


def allocate_curves(spec: ProblemSpec, curves, n_keep, alpha=0.2, steps=40):
    """Budgets [U] int32 from caller-supplied fp32 curves [L][H][T]."""
    L = _lib.lib()
    dev = curves.device
    budgets = torch.empty(spec.units, dtype=torch.int32, device=dev)
    nk = (ctypes.c_int32 * spec.batch)(*[int(x) for x in n_keep])
    # min/max scratch: same layout as the allocation stage's
    ws, n = _workspace(spec, _lib.STAGE_ALLOCATE, dev)
    p = spec.c_problem()
    _check(L.certkv_allocate_curves(ctypes.byref(p), _ptr(curves), nk, float(alpha), int(steps),
                                    _ptr(budgets), _ptr(ws), n, _stream(dev)),
           "certkv_allocate_curves")
    return budgets


def select(spec: ProblemSpec, scores, budgets=None, mode="budget", retain_mass=0.9,
           with_mask=False):
    """(budgets, kept_offsets [U+1] int64, kept_idx int32[, kept_mask [L][H][T] uint8])."""
    L = _lib.lib()
    dev = scores.device
    if mode == "budget":
        assert budgets is not None
        b = budgets.clone()
        cap = int(b.clamp(min=0).sum().item()) if b.numel() else 0
        m = _lib.CERTKV_SELECT_BUDGET
    else:
        b = torch.empty(spec.units, dtype=torch.int32, device=dev)
        cap = spec.layers * spec.kv_heads * spec.total_tokens
        m = _lib.CERTKV_SELECT_COVERAGE
    kept_offsets = torch.empty(spec.units + 1, dtype=torch.int64, device=dev)
    kept_idx = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    mask = torch.empty((spec.layers, spec.kv_heads, spec.total_tokens), dtype=torch.uint8,
                       device=dev) if with_mask else None
    ws, n = _workspace(spec, _lib.STAGE_SELECT, dev)
    p = spec.c_problem()
    _check(L.certkv_select(ctypes.byref(p), _ptr(scores), _ptr(b), m, float(retain_mass),
                           _ptr(kept_offsets), _ptr(kept_idx), cap, _ptr(mask), _ptr(ws), n,
                           _stream(dev)), "certkv_select")
    return (b, kept_offsets, kept_idx, mask) if with_mask else (b, kept_offsets, kept_idx)


def tail_summary(spec: ProblemSpec, scores, k, v, kept_offsets, kept_idx, ksum=None, vsum=None):
    """(k_star [U][d] fp32, v_star [U][d] fp32, tail_mass [U] fp64)."""
    L = _lib.lib()
    dev = k.device
    k_star = torch.empty((spec.units, spec.head_dim), dtype=torch.float32, device=dev)
    v_star = torch.empty_like(k_star)
    tail_mass = torch.empty(spec.units, dtype=torch.float64, device=dev)
    ws, n = _workspace(spec, _lib.STAGE_TAIL, dev)
    p = spec.c_problem()
    _check(L.certkv_tail_summary(ctypes.byref(p), _ptr(scores), _tensor(k), _tensor(v),
                                 _ptr(kept_offsets), _ptr(kept_idx), _ptr(ksum), _ptr(vsum),
                                 _ptr(k_star), _ptr(v_star), _ptr(tail_mass), _ptr(ws), n,
                                 _stream(dev)), "certkv_tail_summary")
    return k_star, v_star, tail_mass


def compact(spec: ProblemSpec, k, v, kept_offsets, kept_idx, k_star, v_star):
    """(k_packed, v_packed [rows][d], pos_packed [rows], packed_offsets [U+1])."""
    L = _lib.lib()
    dev = k.device
    rows = int(kept_offsets[-1].item()) + (spec.units if spec.slot else 0)
    k_packed = torch.empty((rows, spec.head_dim), dtype=k.dtype, device=dev)
    v_packed = torch.empty_like(k_packed)
    pos_packed = torch.empty(rows, dtype=torch.int32, device=dev)
    packed_offsets = torch.empty(spec.units + 1, dtype=torch.int64, device=dev)
    p = spec.c_problem()
    _check(L.certkv_compact(ctypes.byref(p), _tensor(k), _tensor(v), _ptr(kept_offsets),
                            _ptr(kept_idx), _ptr(k_star), _ptr(v_star), _ptr(k_packed),
                            _ptr(v_packed), _ptr(pos_packed), _ptr(packed_offsets), _stream(dev)),
           "certkv_compact")
    return k_packed, v_packed, pos_packed, packed_offsets


def decode_workspace_size(spec: ProblemSpec, tq: int, max_rows: int = 0) -> int:
    p = spec.c_problem()
    return int(_lib.lib().certkv_decode_workspace_size(ctypes.byref(p), int(tq), int(max_rows)))


class DecodeBuffers:
    """Preallocated outputs and workspace of certkv_decode (reusable)."""

    def __init__(self, spec: ProblemSpec, tq: int, device, with_lse=False, max_rows=0):
        self.tq = int(tq)
        self.max_rows = int(max_rows)
        rows = spec.layers * spec.batch * self.tq
        hq = spec.kv_heads * spec.group
        self.out = torch.empty((spec.layers, spec.batch * self.tq, hq, spec.head_dim),
                               dtype=torch.float32, device=device)
        self.lse = torch.empty((spec.layers, spec.batch * self.tq, hq), dtype=torch.float32,
                               device=device) if with_lse else None
        self.ws_bytes = decode_workspace_size(spec, self.tq, self.max_rows)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        assert self.ws.data_ptr() % 256 == 0 and rows > 0


def decode(spec: ProblemSpec, q_new, k_packed, v_packed, packed_offsets, tq, with_lse=False,
           bufs=None, max_rows=0):
    """Attention of tq new queries per sequence (q_new [L][B*tq][Hq][d]) over the packed
    cache: out [L][B*tq][Hq][d] fp32 (and the natural-log lse [L][B*tq][Hq] with_lse).
    max_rows bounds the rows of any head's segment (0: the longest sequence)."""
    L = _lib.lib()
    dev = q_new.device
    if bufs is None:
        bufs = DecodeBuffers(spec, tq, dev, with_lse=with_lse, max_rows=max_rows)
    assert k_packed.is_contiguous() and v_packed.is_contiguous()
    p = spec.c_problem()
    _check(L.certkv_decode(ctypes.byref(p), _tensor(q_new), int(tq), bufs.max_rows, _ptr(k_packed),
                           _ptr(v_packed), _ptr(packed_offsets), _ptr(bufs.out), _ptr(bufs.lse),
                           _ptr(bufs.ws), bufs.ws_bytes, _stream(dev)), "certkv_decode")
    return (bufs.out, bufs.lse) if with_lse else bufs.out


def cluster_tail(spec: ProblemSpec, k, v, perm, budgets, m):
    """Clustered tail summaries: m contiguous groups of each head's evicted
    ranks.  Returns dict(kbar, vbar [U][m][d] in the cache dtype, count [U][m]
    int32, rk, rv [U][m] fp32 radii, vmax_kept [U] fp32)."""
    L = _lib.lib()
    dev = k.device
    U, D = spec.units, spec.head_dim
    out = dict(kbar=torch.empty((U, m, D), dtype=k.dtype, device=dev),
               vbar=torch.empty((U, m, D), dtype=k.dtype, device=dev),
               count=torch.empty((U, m), dtype=torch.int32, device=dev),
               rk=torch.empty((U, m), dtype=torch.float32, device=dev),
               rv=torch.empty((U, m), dtype=torch.float32, device=dev),
               vmax_kept=torch.empty(U, dtype=torch.float32, device=dev))
    p = spec.c_problem()
    _check(L.certkv_cluster_tail(ctypes.byref(p), _tensor(k), _tensor(v), _ptr(perm),
                                 _ptr(budgets), int(m), _ptr(out["kbar"]), _ptr(out["vbar"]),
                                 _ptr(out["count"]), _ptr(out["rk"]), _ptr(out["rv"]),
                                 _ptr(out["vmax_kept"]), _stream(dev)), "certkv_cluster_tail")
    return out


def decode_clustered(spec: ProblemSpec, q_new, k_packed, v_packed, packed_offsets, tq, clusters,
                     max_rows=0):
    """Decode over kept-row segments plus the clustered tail summaries of
    cluster_tail: (out [L][B*tq][Hq][d], lse, bound [L][B*tq][Hq]) fp32, the
    bound being the runtime certificate (inf where it does not hold)."""
    L = _lib.lib()
    dev = q_new.device
    bufs = DecodeBuffers(spec, tq, dev, with_lse=True, max_rows=max_rows)
    bound = torch.empty_like(bufs.lse)
    m = clusters["count"].shape[1]
    p = spec.c_problem()
    _check(L.certkv_decode_clustered(
        ctypes.byref(p), _tensor(q_new), int(tq), bufs.max_rows, _ptr(k_packed), _ptr(v_packed),
        _ptr(packed_offsets), int(m), _ptr(clusters["kbar"]), _ptr(clusters["vbar"]),
        _ptr(clusters["count"]), _ptr(clusters["rk"]), _ptr(clusters["rv"]),
        _ptr(clusters["vmax_kept"]), _ptr(bufs.out), _ptr(bufs.lse), _ptr(bound), _ptr(bufs.ws),
        bufs.ws_bytes, _stream(dev)), "certkv_decode_clustered")
    return bufs.out, bufs.lse, bound


class CompressBuffers:
    """Preallocated outputs and workspace of the fused pass (reusable)."""

    def __init__(self, spec: ProblemSpec, n_keep, device, with_curves=False, with_perm=False,
                 with_mask=False, with_lse=False):
        self.spec = spec
        self.n_keep = [int(x) for x in n_keep]
        H, D = spec.kv_heads, spec.head_dim
        U = spec.units
        slot = 1 if spec.slot else 0
        kept = spec.layers * sum(H * nk - slot * H for nk in self.n_keep)
        rows = kept + slot * U
        shape = (spec.layers, H, spec.total_tokens)
        dt = spec.dtype
        self.scores = torch.empty(shape, dtype=torch.float32, device=device)
        self.budgets = torch.empty(U, dtype=torch.int32, device=device)
        self.kept_offsets = torch.empty(U + 1, dtype=torch.int64, device=device)
        self.kept_idx = torch.empty(max(kept, 1), dtype=torch.int32, device=device)
        self.k_star = torch.empty((U, D), dtype=torch.float32, device=device)
        self.v_star = torch.empty((U, D), dtype=torch.float32, device=device)
        self.tail_mass = torch.empty(U, dtype=torch.float64, device=device)
        self.k_packed = torch.empty((rows, D), dtype=dt, device=device)
        self.v_packed = torch.empty((rows, D), dtype=dt, device=device)
        self.pos_packed = torch.empty(rows, dtype=torch.int32, device=device)
        self.packed_offsets = torch.empty(U + 1, dtype=torch.int64, device=device)
        self.curves = torch.empty(shape, dtype=torch.float32, device=device) if with_curves else None
        self.perm = torch.empty(shape, dtype=torch.int32, device=device) if with_perm else None
        self.alloc_stats = torch.zeros((spec.layers * spec.batch, 3), dtype=torch.int64,
                                       device=device)
        self.kept_mask = torch.empty(shape, dtype=torch.uint8, device=device) if with_mask else None
        self.lse = torch.empty(_lse_shape(spec), dtype=torch.float32, device=device) \
            if with_lse else None
        self.ws, self.ws_bytes = _workspace(spec, _lib.STAGE_COMPRESS, device)
        self._nk = (ctypes.c_int32 * spec.batch)(*self.n_keep)
        self._p = spec.c_problem()
        self._out = _lib.Outputs(*[
            (t.data_ptr() if t is not None else None) for t in (
                self.scores, self.budgets, self.kept_offsets, self.kept_idx, self.k_star,
                self.v_star, self.tail_mass, self.k_packed, self.v_packed, self.pos_packed,
                self.packed_offsets, self.curves, self.perm, self.alloc_stats, self.kept_mask,
                self.lse)])

    def as_dict(self):
        return {k: getattr(self, k) for k in (
            "scores", "budgets", "kept_offsets", "kept_idx", "k_star", "v_star", "tail_mass",
            "k_packed", "v_packed", "pos_packed", "packed_offsets", "curves", "perm",
            "alloc_stats", "kept_mask", "lse")}


def compress(spec: ProblemSpec, q_win, k, v, n_keep, alpha=0.2, steps=40, bufs=None,
             with_curves=False, with_perm=False, with_mask=False, with_lse=False, lse_in=None):
    """The whole pass; returns the CompressBuffers holding every output."""
    L = _lib.lib()
    dev = k.device
    if bufs is None:
        bufs = CompressBuffers(spec, n_keep, dev, with_curves=with_curves, with_perm=with_perm,
                               with_mask=with_mask, with_lse=with_lse)
    if lse_in is not None:
        assert lse_in.dtype == torch.float32 and lse_in.is_contiguous()
        assert tuple(lse_in.shape) == _lse_shape(spec)
    _check(L.certkv_compress(ctypes.byref(bufs._p), _tensor(q_win), _tensor(k), _tensor(v),
                             _ptr(lse_in), bufs._nk, float(alpha), int(steps),
                             ctypes.byref(bufs._out), _ptr(bufs.ws), bufs.ws_bytes, _stream(dev)),
           "certkv_compress")
    return bufs


def profile_enable(on=True):
    _lib.lib().certkv_profile_enable(1 if on else 0)


def profile_reset():
    _lib.lib().certkv_profile_reset()


def profile_read(max_entries=64):
    """{kernel name: (launch count, total ms)} of the launches recorded so far."""
    names = (ctypes.c_char * 64 * max_entries)()
    counts = (ctypes.c_int64 * max_entries)()
    ms = (ctypes.c_double * max_entries)()
    k = _lib.lib().certkv_profile_read(names, counts, ms, max_entries)
    return {names[i].value.decode(): (int(counts[i]), float(ms[i])) for i in range(min(k, max_entries))}
