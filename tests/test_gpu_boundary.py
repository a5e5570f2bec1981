"""GPU tests of the optional parts of the C ABI: the caller's row log-sum-exp
(scoring without the row-sum pass), the row log-sum-exp output, the kept
mask and the device status word for non-finite inputs."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_21541_amd as ck
import synth
from _parity import check_block_stages, score_rel_err, spec_of, unit_id

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _oracle_scores_and_lse(cfg, cache, li, b):
    """Oracle scores [H][n] and the row log-sum-exp laid out [w][Hq] (fp64)."""
    cu = cache["cu_seqlens"]
    n = cu[b + 1] - cu[b]
    H, G, D, w = cfg.kv_heads, cfg.group, cfg.head_dim, cfg.window
    q = cache["q_win"][li, b * w:(b + 1) * w].double().numpy()      # [w][Hq][d]
    k = cache["k"][li, cu[b]:cu[b + 1]].double().numpy()            # [n][H][d]
    qpos = np.repeat(np.arange(n - w, n), G)
    s = np.zeros((H, n))
    lse = np.zeros((w, H * G))
    for h in range(H):
        Q = q[:, h * G:(h + 1) * G].reshape(w * G, D)               # row = q*G + gq
        s[h], lr = oracle.scores(Q, qpos, k[:, h], 1.0 / math.sqrt(D), with_lse=True)
        lse[:, h * G:(h + 1) * G] = lr.reshape(w, G)
    return s, lse


def test_lse_in_and_out_match_oracle():
    cfg = synth.config("C2", seqlens=[4173, 2500])
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg)
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    w, Hq = cfg.window, cfg.kv_heads * cfg.group
    lse_ref = np.zeros((1, cfg.batch * w, Hq))
    s_ref = []
    for b in range(cfg.batch):
        s_b, lse_b = _oracle_scores_and_lse(cfg, cache, 0, b)
        lse_ref[0, b * w:(b + 1) * w] = lse_b
        s_ref.append(s_b)
    # the row log-sum-exp the scorer forms itself
    s_own, lse_out = ck.score(spec, q, k, with_lse=True)
    lse_out = lse_out.cpu().double().numpy()
    err = np.abs(lse_out - lse_ref) / np.maximum(1.0, np.abs(lse_ref))
    log(f"lse_out max error {err.max():.2e}")
    assert err.max() <= 1e-5
    # scoring from the caller's row log-sum-exp (no row-sum pass)
    lse_in = torch.from_numpy(lse_ref.astype(np.float32)).to(dev)
    s_in, lse_echo = ck.score(spec, q, k, lse_in=lse_in, with_lse=True)
    s_in = s_in.cpu().numpy()
    cu = cache["cu_seqlens"]
    for b in range(cfg.batch):
        for h in range(cfg.kv_heads):
            r, sm = score_rel_err(s_in[0, h, cu[b]:cu[b + 1]], s_ref[b][h])
            assert r <= 1e-4 and sm <= 1e-4, (b, h, r, sm)
    # the exported sums are the imported ones to within one rounding each way
    np.testing.assert_allclose(lse_echo.cpu().numpy(), lse_ref.astype(np.float32), rtol=3e-7,
                               atol=1e-7)
    # the fused pass from the caller's row log-sum-exp: every stage against
    # the oracle, end-to-end scores against the oracle's exact ones
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], lse_in=lse_in, with_curves=True,
                       with_perm=True)
    torch.cuda.synchronize()
    out = {name: (t.cpu() if t is not None else None) for name, t in bufs.as_dict().items()}
    for b in range(cfg.batch):
        check_block_stages(spec, cfg, cache, out, 0, b, log=log)


def test_kept_mask_marks_exactly_the_kept_positions():
    cfg = synth.config("C4", seqlens=[3000, 8192 + 5, 1024], layers=2)
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg)
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], with_mask=True)
    torch.cuda.synchronize()
    mask = bufs.kept_mask.cpu().numpy()
    ko = bufs.kept_offsets.cpu().numpy()
    ki = bufs.kept_idx.cpu().numpy()
    cu = cache["cu_seqlens"]
    want = np.zeros_like(mask)
    for li in range(2):
        for b in range(cfg.batch):
            for h in range(cfg.kv_heads):
                u = unit_id(spec, li, b, h)
                want[li, h, cu[b] + ki[ko[u]:ko[u + 1]]] = 1
    assert np.array_equal(mask, want)
    assert int(mask.sum()) == int(bufs.budgets.sum().item())
    # the selection entry point produces the same mask from the same budgets
    _, ko2, ki2, mask2 = ck.select(spec, bufs.scores, bufs.budgets, with_mask=True)
    torch.cuda.synchronize()
    assert np.array_equal(mask2.cpu().numpy(), want)


@pytest.mark.parametrize("where", ["clean", "k_nan", "v_inf", "lse_inf"])
def test_nonfinite_inputs_set_the_status_word(where):
    cfg = synth.config("C2", seqlens=[2000])
    cache = synth.make_cache(cfg, "cpu")
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].clone().to(dev) for x in ("q_win", "k", "v"))
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    spec = ck.ProblemSpec(1, cfg.kv_heads, cfg.group, cfg.head_dim, cfg.window, cfg.seqlens,
                          cfg.dtype, status=status)
    lse_in = None
    if where == "k_nan":
        k[0, 1234, 3, 17] = float("nan")
    elif where == "v_inf":
        v[0, 77, 5, 0] = float("inf")
    elif where == "lse_inf":
        _, lse = ck.score(spec, q, k, with_lse=True)
        lse_in = lse.clone()
        lse_in[0, 5, 9] = float("inf")
        torch.cuda.synchronize()
        assert status.item() == 0
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], lse_in=lse_in)
    torch.cuda.synchronize()
    want = 0 if where == "clean" else ck.CERTKV_ENONFINITE
    assert status.item() == want, (where, status.item())
    # the pass ran to completion and kept its budget algebra
    br, _ = oracle.budget_params(cfg.kv_heads, 2000, cache["n_keep"][0])
    assert int(bufs.budgets.sum().item()) == br


@pytest.mark.parametrize("H,n", [(8, 3000), (64, 40000)])
def test_allocate_curves_with_nonfinite_values_keeps_the_budget_algebra(H, n):
    # Caller curves holding NaN (a whole head, and scattered), +inf and -inf:
    # the status word reports them and the budgets still obey the algebra
    # (each in [b_min, n-1], summing to B_real).  H = 64 with n = 40000 takes
    # the pruned scans and the sequential repair, 8 x 3000 the LDS paths.
    rng = np.random.default_rng(n)
    c = np.abs(np.cumsum(rng.standard_normal((H, n)), 1))[:, ::-1].astype(np.float32)
    c[2, :] = np.nan
    c[4, 100:200] = np.inf
    c[5, 10] = -np.inf
    c[6, ::7] = np.nan
    dev = torch.device("cuda:0")
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    spec = ck.ProblemSpec(1, H, 2, 64, 16, [n], torch.bfloat16, status=status)
    t = torch.from_numpy(np.ascontiguousarray(c)).reshape(1, H, n).to(dev)
    for n_keep in (2, 97, n // 3):
        status.zero_()
        b = ck.allocate_curves(spec, t, [n_keep]).cpu().numpy().reshape(-1)
        torch.cuda.synchronize()
        assert status.item() == ck.CERTKV_ENONFINITE
        br, bm = oracle.budget_params(H, n, n_keep)
        assert int(b.sum()) == br and b.min() >= bm and b.max() <= n - 1, (n_keep, b)


def test_keep_window_matches_oracle():
    # both lengths give b_min >= w = 64 (83 and 70)
    cfg = synth.config("C2", seqlens=[4173, 3500])
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg)
    spec.keep_window = True
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], with_curves=True, with_perm=True)
    torch.cuda.synchronize()
    out = {name: (t.cpu() if t is not None else None) for name, t in bufs.as_dict().items()}
    w, cu = cfg.window, cache["cu_seqlens"]
    ko, ki = out["kept_offsets"].numpy(), out["kept_idx"].numpy()
    for b in range(cfg.batch):
        n = cu[b + 1] - cu[b]
        perm = out["perm"][0, :, cu[b]:cu[b + 1]].numpy()
        assert (perm[:, :w] == np.arange(n - w, n)).all()
        for h in range(cfg.kv_heads):
            u = unit_id(spec, 0, b, h)
            assert set(range(n - w, n)) <= set(ki[ko[u]:ko[u + 1]].tolist())
        check_block_stages(spec, cfg, cache, out, 0, b, log=log, keep_window=True)


def test_keep_window_selection_and_coverage():
    cfg = synth.config("C1")
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg)
    spec.keep_window = True
    dev = torch.device("cuda:0")
    q, k = cache["q_win"].to(dev), cache["k"].to(dev)
    s = ck.score(spec, q, k)
    s_np = s.cpu().numpy()
    n, w, H = cfg.seqlens[0], cfg.window, cfg.kv_heads
    for retain in [0.05, 0.5, 0.9]:
        kb, ko, ki = ck.select(spec, s, mode="coverage", retain_mass=retain)
        torch.cuda.synchronize()
        for h in range(H):
            perm = oracle.order(s_np[0, h], keep_window=w)
            k_eta = oracle.coverage(s_np[0, h], perm, retain, k_min=w)
            assert kb[h].item() == k_eta, (retain, h, kb[h].item(), k_eta)
            kept = ki[ko[h].item():ko[h + 1].item()].cpu().numpy()
            assert np.array_equal(kept, oracle.select(perm, k_eta))
    # a caller budget below w keeps the first window keys; above it, the
    # window plus the best of the rest
    for bsel in [5, w, w + 37]:
        bud = torch.full((H,), bsel, dtype=torch.int32, device=dev)
        _, ko, ki = ck.select(spec, s, bud)
        torch.cuda.synchronize()
        for h in range(H):
            perm = oracle.order(s_np[0, h], keep_window=w)
            kept = ki[ko[h].item():ko[h + 1].item()].cpu().numpy()
            assert np.array_equal(kept, oracle.select(perm, bsel)), (bsel, h)
