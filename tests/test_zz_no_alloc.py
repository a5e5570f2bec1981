"""The no-allocation scoring entry point (certkv_score_noalloc, workspace in
the library's fixed device array) against certkv_score, through the C ABI:
identical kernels on identical inputs, so identical bits, on two calls in a
row, the second with a smaller problem (the array keeps the first call's
contents)."""
import ctypes

import pytest
import torch

import paper_2608_21541_amd as ck
import synth
from paper_2608_21541_amd import _lib
from _parity import spec_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _case(seqlens, layers, with_lse_in=False):
    cfg = synth.config("C2", seqlens=seqlens, layers=layers)
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg)
    dev = torch.device("cuda:0")
    q, k = cache["q_win"].to(dev), cache["k"].to(dev)
    lse_in = None
    if with_lse_in:
        _, lse_in = ck.score(spec, q, k, with_lse=True)
    s_ref, ksum_ref, lse_ref = ck.score(spec, q, k, with_ksum=True, with_lse=True, lse_in=lse_in)
    scores = torch.empty_like(s_ref)
    ksum = torch.empty_like(ksum_ref)
    lse = torch.empty_like(lse_ref)
    ck.score_noalloc(spec, q, k, scores, ksum=ksum, lse_out=lse, lse_in=lse_in)
    torch.cuda.synchronize()
    assert torch.equal(scores, s_ref)
    assert torch.equal(ksum, ksum_ref)
    assert torch.equal(lse, lse_ref)
    return scores


def test_noalloc_score_matches_score_on_two_calls():
    # first a two-layer ragged batch at the 8B head shapes, then a smaller
    # single-layer problem that reuses the array
    big = _case([32768, 9001], 2)
    small = _case([3001], 1)
    assert big.numel() > small.numel()
    # and with the caller's row log-sum-exp (pass 1 skipped)
    _case([5000], 1, with_lse_in=True)


def test_noalloc_rejects_a_workspace_beyond_the_array():
    L = _lib.lib()
    cap = L.certkv_score_noalloc_max_bytes()
    assert cap == 64 << 20
    # 160 layers x 64 KV heads x 8-way groups at 131072 tokens: the scoring
    # partials alone exceed the array
    n = 131072
    cu = (ctypes.c_int64 * 2)(0, n)
    p = _lib.Problem(160, 1, 64, 8, 128, 64, ctypes.cast(cu, ctypes.POINTER(ctypes.c_int64)),
                     _lib.CERTKV_BF16, _lib.CERTKV_BF16, 0.0,
                     _lib.CERTKV_CAUSAL | _lib.CERTKV_DRY_RUN, None)
    assert L.certkv_workspace_size(ctypes.byref(p), _lib.STAGE_SCORE) > cap
    t = _lib.Tensor(1 << 20, 64 * 128 * n, 64 * 128, 128)
    assert L.certkv_score_noalloc(ctypes.byref(p), t, t, None, 1 << 20, None, None,
                                  None) == _lib.CERTKV_EWORKSPACE
