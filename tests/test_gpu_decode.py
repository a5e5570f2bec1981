"""GPU parity of decode over the packed cache (certkv_decode) against the
oracle, the keep-all identity, and the future-query lift bound evaluated on
the GPU's outputs."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_21541_amd as ck
import synth
from _parity import spec_of, unit_id

pytestmark = pytest.mark.gpu

OUT_RTOL = 1e-4   # relative L2 per output row (fp32 accumulation, 16-bit weight split)
LSE_ATOL = 1e-4


def log(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _compress(cfg, cache, n_keep=None):
    spec = spec_of(cfg, layers=len(cache["layers"]))
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    bufs = ck.compress(spec, q, k, v, cache["n_keep"] if n_keep is None else n_keep)
    torch.cuda.synchronize()
    return spec, bufs


def _row_err(x, ref):
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-30))


def _check_against_oracle(cfg, cache, spec, bufs, tq, seed_offset=7919):
    dev = torch.device("cuda:0")
    qn = synth.make_queries(cfg, tq, "cpu", layers=cache["layers"], seed_offset=seed_offset)
    out, lse = ck.decode(spec, qn.to(dev), bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq,
                         with_lse=True)
    torch.cuda.synchronize()
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    kp = bufs.k_packed.cpu().double().numpy()
    vp = bufs.v_packed.cpu().double().numpy()
    po = bufs.packed_offsets.cpu().numpy()
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    scale = 1.0 / math.sqrt(D)
    worst, worst_lse = 0.0, 0.0
    for li in range(len(cache["layers"])):
        for b in range(cfg.batch):
            for h in range(H):
                u = unit_id(spec, li, b, h)
                seg = slice(po[u], po[u + 1])
                q = qn[li, b * tq:(b + 1) * tq, h * G:(h + 1) * G].double().numpy().reshape(-1, D)
                ref, ref_lse = oracle.decode(q, kp[seg], vp[seg], scale)
                got = out[li, b * tq:(b + 1) * tq, h * G:(h + 1) * G].reshape(-1, D)
                got_lse = lse[li, b * tq:(b + 1) * tq, h * G:(h + 1) * G].reshape(-1)
                for r in range(tq * G):
                    e = _row_err(got[r], ref[r])
                    assert e <= OUT_RTOL, (li, b, h, r, e)
                    worst = max(worst, e)
                d_lse = np.abs(got_lse - ref_lse).max()
                assert d_lse <= LSE_ATOL, (li, b, h, d_lse)
                worst_lse = max(worst_lse, float(d_lse))
    log(f"decode tq={tq}: worst row error {worst:.2e}, worst lse error {worst_lse:.2e}")
    return out


@pytest.mark.parametrize("tq", [1, 8, 33, 65])
def test_decode_matches_oracle_ragged_batch(tq):
    # ragged lengths (segments of varying length, ragged last tiles), two
    # layers; tq = 33 gives 132 query rows (a padded fifth 32-row tile), tq = 65
    # gives 260 rows (sixteen query tiles, the largest workgroup)
    cfg = synth.config("C4", seqlens=[3000, 8192 + 5, 1024], layers=2)
    cache = synth.make_cache(cfg, "cpu")
    spec, bufs = _compress(cfg, cache)
    _check_against_oracle(cfg, cache, spec, bufs, tq)


@pytest.mark.parametrize("tq", [1, 40, 130])
def test_decode_head_dim_64_without_grouping(tq):
    # head_dim 64, one query head per KV head (G = 1): one, two and eight
    # query tiles (the first two split the output dims over two waves)
    cfg = synth.config("C1", seqlens=[3000, 1500])
    cfg.dtype = torch.bfloat16
    cache = synth.make_cache(cfg, "cpu")
    spec, bufs = _compress(cfg, cache)
    _check_against_oracle(cfg, cache, spec, bufs, tq)


@pytest.mark.parametrize("tq", [1, 16])
def test_decode_cancelling_pairs(tq):
    # the 70B-class shape (G = 8) with 256 cancelling value pairs per head:
    # evicted pairs whose values cancel leave a slot value near zero while
    # their keys keep mass; decode over that cache against the oracle
    cfg = synth.config("C5", seqlens=[6000, 2500], layers=1)
    cache = synth.make_cache(cfg, "cpu")
    spec, bufs = _compress(cfg, cache)
    _check_against_oracle(cfg, cache, spec, bufs, tq)


def test_keep_all_decode_equals_full_attention():
    # n_keep = n: every head keeps n - 1 real rows and its slot is the one
    # evicted key itself, so decode over the packed cache is exact attention
    # over the whole cache.
    # 9037 keys: segments of three 4096-key chunks with a ragged last tile
    cfg = synth.config("C2", seqlens=[9037])
    cache = synth.make_cache(cfg, "cpu")
    n = cfg.seqlens[0]
    spec, bufs = _compress(cfg, cache, n_keep=[n])
    tq = 4
    dev = torch.device("cuda:0")
    qn = synth.make_queries(cfg, tq, "cpu")
    out = ck.decode(spec, qn.to(dev), bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    k = cache["k"][0].double().numpy()
    v = cache["v"][0].double().numpy()
    for h in range(H):
        q = qn[0, :, h * G:(h + 1) * G].double().numpy().reshape(-1, D)
        ref, _ = oracle.decode(q, k[:, h], v[:, h], 1.0 / math.sqrt(D))
        got = out[0, :, h * G:(h + 1) * G].reshape(-1, D)
        for r in range(tq * G):
            assert _row_err(got[r], ref[r]) <= OUT_RTOL, (h, r)


@pytest.mark.parametrize("name", ["C2", "C5"])
def test_future_query_lift_bound_on_gpu_outputs(name):
    # The a-posteriori bound of the future-query lift theorem with the GPU's
    # compressed output: ||O - Ohat|| <= V_max (2 |p - q| + min(p, q) ||a - r||_1)
    # + q ||v*_stored - sum_T r_j v_j|| (the stored slot is rounded to bf16).
    cfg = synth.config(name, seqlens=[4000], layers=1)
    cache = synth.make_cache(cfg, "cpu")
    spec, bufs = _compress(cfg, cache)
    tq = 4
    dev = torch.device("cuda:0")
    qn = synth.make_queries(cfg, tq, "cpu")
    out = ck.decode(spec, qn.to(dev), bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    scale = 1.0 / math.sqrt(D)
    n = cfg.seqlens[0]
    k = cache["k"][0].double().numpy()
    v = cache["v"][0].double().numpy()
    s = bufs.scores[0].cpu().double().numpy()
    ko, ki = bufs.kept_offsets.cpu().numpy(), bufs.kept_idx.cpu().numpy()
    po = bufs.packed_offsets.cpu().numpy()
    kp = bufs.k_packed.cpu().double().numpy()
    vp = bufs.v_packed.cpu().double().numpy()
    worst_ratio = 0.0
    for h in range(H):
        u = unit_id(spec, 0, 0, h)
        kept = np.zeros(n, bool)
        kept[ki[ko[u]:ko[u + 1]]] = True
        r = np.where(kept, 0.0, np.maximum(s[h], 0.0))
        r /= r.sum()
        kslot, vslot = kp[po[u + 1] - 1], vp[po[u + 1] - 1]
        slack_v = np.linalg.norm(vslot - r @ v[:, h])
        for row in range(tq * G):
            t, g = divmod(row, G)
            q = qn[0, t, h * G + g].double().numpy()
            terms = oracle.lift_terms(q, k[:, h], v[:, h], kept, r, kslot, vslot, scale)
            # the exact output from the oracle, the compressed one from the GPU
            o_full, _ = oracle.decode(q[None], k[:, h], v[:, h], scale)
            err_gpu = float(np.linalg.norm(out[0, t, h * G + g] - o_full[0]))
            bound = terms["v_max"] * (2 * abs(terms["p"] - terms["q"]) +
                                      min(terms["p"], terms["q"]) * terms["l1"])
            bound += terms["q"] * slack_v + 1e-4 * np.linalg.norm(o_full[0])
            assert err_gpu <= bound, (h, row, err_gpu, bound, terms)
            assert abs(terms["p"] - terms["q"]) <= math.tanh(
                abs(terms["lam_T"] - terms["z_slot"]) / 4) + 1e-12
            worst_ratio = max(worst_ratio, err_gpu / bound)
    log(f"lift bound: worst ||O - Ohat|| / bound = {worst_ratio:.3f}")


def test_keep_all_segment_of_exactly_one_chunk():
    # n = 4096 with n_keep = n: every head's segment (n - 1 kept rows and the
    # slot) fills exactly one 4096-key chunk, which is also the default row
    # bound of the workspace.
    cfg = synth.config("C2", seqlens=[4096])
    cache = synth.make_cache(cfg, "cpu")
    n = cfg.seqlens[0]
    spec, bufs = _compress(cfg, cache, n_keep=[n])
    po = bufs.packed_offsets.cpu().numpy()
    log(f"segment rows {np.diff(po).max()}")
    _check_against_oracle(cfg, cache, spec, bufs, tq=2)


def test_decode_row_bound_gives_same_output_and_flags_overflow():
    # keep-all segments of 9036 and 5999 rows: three and two 4096-key chunks
    cfg = synth.config("C4", seqlens=[9037, 6000])
    cache = synth.make_cache(cfg, "cpu")
    spec, bufs = _compress(cfg, cache, n_keep=list(cfg.seqlens))
    dev = torch.device("cuda:0")
    tq = 8
    qn = synth.make_queries(cfg, tq, "cpu").to(dev)
    seg = int(np.diff(bufs.packed_offsets.cpu().numpy()).max())
    log(f"longest segment {seg} rows")
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    spec.status = status
    ref = ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq)
    tight = ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq,
                      max_rows=seg)
    torch.cuda.synchronize()
    assert int(status.item()) == ck.CERTKV_OK
    # the same 4096-key chunks in the same order: the same bits
    assert torch.equal(ref, tight)
    assert ck.decode_workspace_size(spec, tq, seg - 4096) < ck.decode_workspace_size(spec, tq)
    # a bound below the longest segment (by more than a chunk) is reported
    ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq,
              max_rows=seg - 4096)
    torch.cuda.synchronize()
    assert int(status.item()) == ck.CERTKV_ERANGE
