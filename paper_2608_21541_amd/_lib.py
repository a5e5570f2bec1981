"""ctypes view of libcertkv.so (the C ABI declared in include/certkv.h).

The library is loaded from this package directory only.  There is no
fallback: if the shared library is missing the import of any compute entry
point raises, so nothing can silently run elsewhere.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcertkv.so")

CERTKV_OK = 0
CERTKV_EINVAL = -1
CERTKV_EUNSUPPORTED = -2
CERTKV_EINFEASIBLE = -3
CERTKV_ENONFINITE = -4
CERTKV_EWORKSPACE = -5
CERTKV_EHIP = -6
CERTKV_ERANGE = -7

CERTKV_F32 = 0
CERTKV_BF16 = 1
CERTKV_CAUSAL = 1
CERTKV_DRY_RUN = 2
CERTKV_KEEP_WINDOW = 4
CERTKV_STAT_UNCENTERED = 1 << 3
CERTKV_STAT_TAIL_MASS = 1 << 4
CERTKV_ALLOC_UNIFORM = 1 << 5
CERTKV_ALLOC_GREEDY = 1 << 6
CERTKV_NO_SLOT = 1 << 7
CERTKV_SELECT_BUDGET = 0
CERTKV_SELECT_COVERAGE = 1

STAGE_SCORE = 1
STAGE_ALLOCATE = 2
STAGE_SELECT = 3
STAGE_TAIL = 4
STAGE_COMPACT = 5
STAGE_COMPRESS = 6

EXPORTS = [
    "certkv_status_string", "certkv_workspace_size", "certkv_score", "certkv_allocate",
    "certkv_allocate_curves", "certkv_select", "certkv_tail_summary", "certkv_compact",
    "certkv_compress", "certkv_decode_workspace_size", "certkv_decode", "certkv_cluster_tail",
    "certkv_decode_clustered", "certkv_profile_enable",
    "certkv_profile_read", "certkv_profile_reset",
    "certkv_score_noalloc", "certkv_score_noalloc_max_bytes",
]


class Problem(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("cu_seqlens_host", ctypes.POINTER(ctypes.c_int64)),
        ("q_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("flags", ctypes.c_uint32),
        ("dev_status", ctypes.c_void_p),
    ]


class Tensor(ctypes.Structure):
    _fields_ = [
        ("ptr", ctypes.c_void_p),
        ("s_layer", ctypes.c_int64),
        ("s_token", ctypes.c_int64),
        ("s_head", ctypes.c_int64),
    ]


class Outputs(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in (
        "scores", "budgets", "kept_offsets", "kept_idx", "k_star", "v_star", "tail_mass",
        "k_packed", "v_packed", "pos_packed", "packed_offsets", "curves", "perm", "alloc_stats",
        "kept_mask", "lse")]


class CertKVError(RuntimeError):
    def __init__(self, status, what):
        msg = _LIB.certkv_status_string(status).decode() if _LIB is not None else str(status)
        super().__init__(f"{what}: {msg} (status {status})")
        self.status = status


_LIB = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"libcertkv.so not found at {LIB_PATH}; build it first "
            "(python -m paper_2608_21541_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(Problem)
    vp, i32, i64, dbl, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t
    L.certkv_status_string.argtypes = [i32]
    L.certkv_status_string.restype = ctypes.c_char_p
    L.certkv_workspace_size.argtypes = [P, i32]
    L.certkv_workspace_size.restype = sz
    L.certkv_score.argtypes = [P, Tensor, Tensor, vp, vp, vp, vp, vp, sz, vp]
    L.certkv_score_noalloc.argtypes = [P, Tensor, Tensor, vp, vp, vp, vp, vp]
    L.certkv_score_noalloc_max_bytes.argtypes = []
    L.certkv_score_noalloc_max_bytes.restype = sz
    L.certkv_allocate.argtypes = [P, vp, Tensor, vp, dbl, i32, vp, vp, vp, vp, vp, sz, vp]
    L.certkv_allocate_curves.argtypes = [P, vp, vp, dbl, i32, vp, vp, sz, vp]
    L.certkv_select.argtypes = [P, vp, vp, i32, dbl, vp, vp, i64, vp, vp, sz, vp]
    L.certkv_tail_summary.argtypes = [P, vp, Tensor, Tensor, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.certkv_compact.argtypes = [P, Tensor, Tensor, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.certkv_compress.argtypes = [P, Tensor, Tensor, Tensor, vp, vp, dbl, i32,
                                  ctypes.POINTER(Outputs), vp, sz, vp]
    L.certkv_decode_workspace_size.argtypes = [P, i32, i32]
    L.certkv_decode_workspace_size.restype = sz
    L.certkv_decode.argtypes = [P, Tensor, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]
    L.certkv_cluster_tail.argtypes = [P, Tensor, Tensor, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp]
    L.certkv_decode_clustered.argtypes = [P, Tensor, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp,
                                          vp, vp, vp, vp, vp, vp, sz, vp]
    L.certkv_profile_enable.argtypes = [i32]
    L.certkv_profile_read.argtypes = [vp, vp, vp, i32]
    L.certkv_profile_read.restype = i32
    L.certkv_profile_reset.argtypes = []
    L.certkv_profile_reset.restype = None
    for name in EXPORTS:
        if name not in ("certkv_status_string", "certkv_workspace_size",
                        "certkv_decode_workspace_size", "certkv_profile_read",
                        "certkv_profile_reset", "certkv_score_noalloc_max_bytes"):
            getattr(L, name).restype = i32
    _LIB = L
    return L
