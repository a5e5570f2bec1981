"""Shared helpers of the GPU parity tests: run the HIP path on a synthetic
cache and compare one (layer, sequence) block with the CPU oracle."""
import math

import numpy as np
import torch

import oracle
import paper_2608_21541_amd as ck
import synth

# Tolerances (the workload's own: per-key mass 1e-4 relative, slot vectors
# and reconstructed window outputs 2e-3 relative L2).
SCORE_RTOL = 1e-4
VEC_RTOL = 2e-3


def spec_of(cfg, layers=None):
    return ck.ProblemSpec(cfg.layers if layers is None else layers, cfg.kv_heads, cfg.group,
                          cfg.head_dim, cfg.window, list(cfg.seqlens), cfg.dtype)


def run_gpu(cfg, cache, with_extras=True):
    spec = spec_of(cfg, layers=len(cache["layers"]))
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], with_curves=with_extras,
                       with_perm=with_extras)
    torch.cuda.synchronize()
    out = {name: (t.cpu() if t is not None else None) for name, t in bufs.as_dict().items()}
    return spec, out, (q, k, v), bufs


def to_np64(t):
    return t.to(torch.float64).cpu().numpy()


def block_inputs(cache, li, b):
    """(q [w][Hq][d], k [n][H][d], v [n][H][d]) of layer index li, sequence b, fp64."""
    cfg = cache["cfg"]
    cu = cache["cu_seqlens"]
    w = cfg.window
    q = to_np64(cache["q_win"][li, b * w:(b + 1) * w])
    k = to_np64(cache["k"][li, cu[b]:cu[b + 1]])
    v = to_np64(cache["v"][li, cu[b]:cu[b + 1]])
    return q, k, v


def unit_id(spec, l, b, h):
    return (l * spec.batch + b) * spec.kv_heads + h


def score_rel_err(s_gpu, s_ref):
    s_gpu = np.asarray(s_gpu, np.float64)
    floor = 1e-30 * s_ref.max()
    big = s_ref >= floor
    rel = np.abs(s_gpu[big] - s_ref[big]) / s_ref[big]
    small_abs = np.abs(s_gpu[~big] - s_ref[~big]).max() if (~big).any() else 0.0
    return float(rel.max()), float(small_abs / max(s_ref.max(), 1e-300))


def vec_rel_err(x, ref, scale):
    return float(np.linalg.norm(np.asarray(x, np.float64) - ref) / max(np.linalg.norm(ref), scale,
                                                                       1e-300))


def check_block_stages(spec, cfg, cache, out, li, b, check_scores=True, log=print,
                       keep_window=False, alpha=0.2, statistic="centered",
                       allocator="lagrangian", slot=True):
    """Compare one (layer, sequence) block of the GPU output with the oracle.

    Integer stages are compared against the oracle fed the GPU's own upstream
    arrays (scores for order/select, curves for the allocation): bit-exact.
    Floating outputs are compared to the workload's tolerances.  Returns a
    dict of measured errors.
    """
    cu = cache["cu_seqlens"]
    n = cu[b + 1] - cu[b]
    H, D, w, G = cfg.kv_heads, cfg.head_dim, cfg.window, cfg.group
    t0, t1 = cu[b], cu[b + 1]
    q, k, v = block_inputs(cache, li, b)
    scale = 1.0 / math.sqrt(D)
    s_gpu = out["scores"][li, :, t0:t1].numpy()            # [H][n]
    perm_gpu = out["perm"][li, :, t0:t1].numpy()
    c_gpu = out["curves"][li, :, t0:t1].numpy()
    units = [unit_id(spec, li, b, h) for h in range(H)]
    bud_gpu = out["budgets"].numpy()[units]
    n_keep = cache["n_keep"][b]
    res = {}

    # Stage parity: the oracle's steps fed the GPU scores.
    var = dict(statistic=statistic, allocator=allocator, slot=slot)
    st = oracle.compress_block(q, k, v, n_keep, scale, s32_in=s_gpu, keep_window=keep_window,
                               alpha=alpha, **var)
    assert np.array_equal(st["perm"], perm_gpu), "order differs from the oracle's on the same scores"
    dc = np.abs(c_gpu.astype(np.float64) - st["c32"].astype(np.float64))
    cmax = float(st["c32"].max())
    tol_c = 4.0 * np.spacing(np.abs(st["c32"])).astype(np.float64) + 1e-6 * cmax
    assert (dc <= tol_c).all(), f"curves off by {dc.max()} (max c {cmax})"
    res["curve_bits_differ"] = int((c_gpu != st["c32"]).sum())
    b_on_gpu_curves, _ = oracle.allocate(c_gpu, n_keep, alpha=alpha, allocator=allocator,
                                         slot=slot)
    assert np.array_equal(b_on_gpu_curves, bud_gpu), (b_on_gpu_curves, bud_gpu)
    res["budgets_equal_oracle_curves"] = bool(np.array_equal(st["budgets"], bud_gpu))
    br, bm = oracle.budget_params(H, n, n_keep, alpha, slot=slot)
    assert int(bud_gpu.sum()) == br and bud_gpu.min() >= bm and bud_gpu.max() <= n - 1

    ko = out["kept_offsets"].numpy()
    po = out["packed_offsets"].numpy()
    kept_all = out["kept_idx"].numpy()
    kp = out["k_packed"]
    vp = out["v_packed"]
    pos = out["pos_packed"].numpy()
    k_src = cache["k"][li, t0:t1]
    v_src = cache["v"][li, t0:t1]
    worst_vec = 0.0
    worst_rec = 0.0
    for h, u in enumerate(units):
        kept = kept_all[ko[u]:ko[u + 1]]
        assert len(kept) == bud_gpu[h]
        ref_kept = oracle.select(perm_gpu[h], bud_gpu[h])
        assert np.array_equal(kept, ref_kept), f"kept set of head {h} differs"
        ks, vs, m = oracle.tail(s_gpu[h], kept, k[:, h], v[:, h])
        a = oracle.normalize(s_gpu[h])
        mask = np.zeros(n, bool)
        mask[kept] = True
        ME_k = float((a[~mask] * np.linalg.norm(k[~mask, h], axis=1)).sum()) / max(m, 1e-300)
        ME_v = float((a[~mask] * np.linalg.norm(v[~mask, h], axis=1)).sum()) / max(m, 1e-300)
        ek = vec_rel_err(out["k_star"][u].numpy(), ks, ME_k)
        ev = vec_rel_err(out["v_star"][u].numpy(), vs, ME_v)
        assert ek <= VEC_RTOL and ev <= VEC_RTOL, (h, ek, ev)
        assert abs(out["tail_mass"][u].item() - m) <= 1e-9 * max(m, 1e-30) + 1e-15
        worst_vec = max(worst_vec, ek, ev)
        # pooled window output reproduced by kept rows + m * v*
        full = (a[:, None] * v[:, h]).sum(0)
        err = oracle.row_error(a, v[:, h], mask, m * out["v_star"][u].numpy().astype(np.float64))
        rec = err / max(np.linalg.norm(full), ME_v * m, 1e-300)
        assert rec <= VEC_RTOL, (h, rec)
        worst_rec = max(worst_rec, rec)
        # packed segment: kept rows copied bit-exactly, then the rounded slot
        # (no slot row without the slot)
        p0, p1 = po[u], po[u + 1]
        pk = p1 - 1 if slot else p1
        assert pk - p0 == len(kept)
        assert np.array_equal(pos[p0:pk], kept)
        assert torch.equal(kp[p0:pk], k_src[kept, h].cpu()) and \
            torch.equal(vp[p0:pk], v_src[kept, h].cpu())
        if slot:
            assert pos[p1 - 1] == -1
            slot_k = out["k_star"][u].to(kp.dtype)
            slot_v = out["v_star"][u].to(vp.dtype)
            assert torch.equal(kp[p1 - 1], slot_k) and torch.equal(vp[p1 - 1], slot_v)
    res["worst_slot_err"] = worst_vec
    res["worst_pooled_err"] = worst_rec
    blk = po[units[-1] + 1] - po[units[0]]
    assert blk == H * n_keep, "packed rows per (layer, sequence) must equal H * n_keep"

    if check_scores:
        e2e = oracle.compress_block(q, k, v, n_keep, scale, keep_window=keep_window,
                                    alpha=alpha, **var)
        worst = 0.0
        for h in range(H):
            r, sm = score_rel_err(s_gpu[h], e2e["s"][h])
            assert r <= SCORE_RTOL and sm <= SCORE_RTOL, (h, r, sm)
            worst = max(worst, r)
            assert abs(s_gpu[h].astype(np.float64).sum() - w * G) <= 1e-4 * w * G
        res["worst_score_rel"] = worst
        res["e2e_budgets_equal"] = bool(np.array_equal(e2e["budgets"], bud_gpu))
    log(f"block layer {li} seq {b}: {res}")
    return res
