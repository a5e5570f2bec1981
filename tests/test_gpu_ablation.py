"""GPU parity of the one-factor ablation variants (statistic, allocator, no
slot, safeguard alpha) against the oracle's branches, through the C ABI."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_21541_amd as ck
import synth
from _parity import check_block_stages, spec_of, unit_id

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


VARIANTS = [
    ("tail_mass", dict(statistic="tail_mass")),
    ("uncentered", dict(statistic="uncentered")),
    ("uniform", dict(allocator="uniform")),
    ("greedy", dict(allocator="greedy")),
    ("no_slot", dict(slot=False)),
    ("alpha_0", dict(alpha=0.0)),
    ("alpha_0.4", dict(alpha=0.4)),
    ("snapkv_uniform", dict(allocator="uniform", slot=False)),
]


def _run(var, seqlens=(6000, 2049)):
    cfg = synth.config("C2", seqlens=list(seqlens), layers=1)
    cache = synth.make_cache(cfg, "cpu")
    spec = spec_of(cfg, layers=1)
    spec.statistic = var.get("statistic", "centered")
    spec.allocator = var.get("allocator", "lagrangian")
    spec.slot = var.get("slot", True)
    dev = torch.device("cuda:0")
    q, k, v = (cache[x].to(dev) for x in ("q_win", "k", "v"))
    bufs = ck.compress(spec, q, k, v, cache["n_keep"], alpha=var.get("alpha", 0.2),
                       with_curves=True, with_perm=True)
    torch.cuda.synchronize()
    out = {name: (t.cpu() if t is not None else None) for name, t in bufs.as_dict().items()}
    return cfg, cache, spec, out, bufs, (q, k, v)


@pytest.mark.parametrize("name,var", VARIANTS, ids=[n for n, _ in VARIANTS])
def test_variant_matches_oracle(name, var):
    cfg, cache, spec, out, _, _ = _run(var)
    log(f"variant {name}")
    for b in range(cfg.batch):
        check_block_stages(spec, cfg, cache, out, 0, b, log=log, alpha=var.get("alpha", 0.2),
                           statistic=var.get("statistic", "centered"),
                           allocator=var.get("allocator", "lagrangian"),
                           slot=var.get("slot", True))
    if var.get("allocator") == "uniform":
        slot = var.get("slot", True)
        for b in range(cfg.batch):
            units = [unit_id(spec, 0, b, h) for h in range(cfg.kv_heads)]
            want = cache["n_keep"][b] - (1 if slot else 0)
            assert (out["budgets"].numpy()[units] == want).all()


def test_no_slot_stage_entry_points_and_decode():
    # the standalone compaction lays out the same slot-free segments as the
    # fused pass, and decode attends over the kept rows alone
    cfg, cache, spec, out, bufs, (q, k, v) = _run(dict(slot=False), seqlens=(3000,))
    kp, vp, pos, po = ck.compact(spec, k, v, bufs.kept_offsets, bufs.kept_idx, bufs.k_star,
                                 bufs.v_star)
    torch.cuda.synchronize()
    assert torch.equal(po.cpu(), out["packed_offsets"])
    assert torch.equal(kp.cpu(), out["k_packed"]) and torch.equal(vp.cpu(), out["v_packed"])
    assert torch.equal(pos.cpu(), out["pos_packed"])
    assert int(po[-1]) == int(bufs.kept_offsets[-1])
    tq = 3
    qn = synth.make_queries(cfg, tq, "cpu")
    o = ck.decode(spec, qn.to(k.device), bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq)
    torch.cuda.synchronize()
    o = o.cpu().numpy()
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    ko = out["kept_offsets"].numpy()
    ki = out["kept_idx"].numpy()
    kc, vc = cache["k"][0].double().numpy(), cache["v"][0].double().numpy()
    for h in range(H):
        u = unit_id(spec, 0, 0, h)
        kept = ki[ko[u]:ko[u + 1]]
        qh = qn[0, :, h * G:(h + 1) * G].double().numpy().reshape(-1, D)
        ref, _ = oracle.decode(qh, kc[kept, h], vc[kept, h], 1.0 / math.sqrt(D))
        got = o[0, :, h * G:(h + 1) * G].reshape(-1, D)
        err = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
        assert err.max() <= 1e-4, (h, err.max())
