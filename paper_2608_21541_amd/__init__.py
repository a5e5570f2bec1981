"""CertKV one-shot KV-cache compression for MI355X (gfx950).

The compute path is libcertkv.so (HIP kernels behind a C ABI, see
include/certkv.h); this package holds the build script and a thin ctypes
binding with the same entry-point names.
"""
from .api import (ProblemSpec, CompressBuffers, score, score_noalloc, allocate, allocate_curves, select,  # noqa: F401
                  tail_summary, compact, compress, workspace_size, decode, DecodeBuffers,
                  decode_workspace_size, cluster_tail, decode_clustered, profile_enable, profile_reset, profile_read)
from ._lib import CertKVError, CERTKV_OK, CERTKV_ENONFINITE, CERTKV_ERANGE  # noqa: F401
