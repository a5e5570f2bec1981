"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times: the 32-layer Llama-3-8B-shaped cache at 131072 tokens and the
80-layer Llama-3-70B-shaped one.

Every layer is compared with the oracle.  Algorithm 1 runs independently per
(layer, sequence), so the stage parity of each layer is the oracle fed that
layer's GPU scores (order, kept sets, packed layout bit-exact; budgets
bit-exact on the GPU's curves; curves and slot vectors to tolerance).
End-to-end scores (the oracle's own fp64 scoring) are compared on four layers
spread over the depth.  Decode over the full packed cache has more work items
than the persistent grid has workgroups, so each workgroup runs several items;
it is compared with the oracle on sampled heads including the longest segment.
"""
import concurrent.futures
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_21541_amd as ck
import synth
from _parity import check_block_stages, score_rel_err, spec_of, unit_id

pytestmark = pytest.mark.gpu

LAYER_CHUNK = 8        # layers per test (the oracle on 8 full layers takes ~20-40 s)
DEC_KEYS = 4096        # keys per decode work item
DEC_WG_PER_CU = 2      # resident decode workgroups per CU (80 KiB of LDS stages each)


def log(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


@pytest.fixture(scope="module", params=["C3", "C5"])
def full(request):
    name = request.param
    cfg = synth.config(name)
    log(f"{name}: generating {cfg.layers} layers on the GPU")
    cache = synth.make_cache(cfg, "cuda:0")
    spec = spec_of(cfg)
    bufs = ck.compress(spec, cache["q_win"], cache["k"], cache["v"], cache["n_keep"],
                       with_curves=True, with_perm=True)
    torch.cuda.synchronize()
    out = {k: (t.cpu() if t is not None else None) for k, t in bufs.as_dict().items()}
    # the oracle reads the same tensors (each layer is copied to the host, in
    # fp64, when it is checked)
    yield dict(name=name, cfg=cfg, cache=cache, spec=spec, bufs=bufs, out=out)
    del bufs, cache
    torch.cuda.empty_cache()


def _chunks(layers):
    return [list(range(i, min(i + LAYER_CHUNK, layers))) for i in range(0, layers, LAYER_CHUNK)]


def test_full_size_invariants(full):
    cfg, spec, out, cache = full["cfg"], full["spec"], full["out"], full["cache"]
    L, H = spec.layers, cfg.kv_heads
    w, G = cfg.window, cfg.group
    s = out["scores"].to(torch.float64)
    cu = cache["cu_seqlens"]
    for b in range(cfg.batch):
        tot = s[:, :, cu[b]:cu[b + 1]].sum(-1)
        assert torch.all((tot - w * G).abs() <= 1e-3 * w * G)
    bud = out["budgets"].numpy().reshape(L, cfg.batch, H)
    for b in range(cfg.batch):
        br, bm = oracle.budget_params(H, cu[b + 1] - cu[b], cache["n_keep"][b])
        assert (bud[:, b].sum(-1) == br).all() and bud[:, b].min() >= bm
    po = out["packed_offsets"].numpy()
    ko = out["kept_offsets"].numpy()
    assert (po - ko == np.arange(len(po))).all()
    assert (np.diff(ko) == out["budgets"].numpy()).all()
    assert (out["tail_mass"].numpy() > 0).all()


# Stage parity on every layer: chunks of LAYER_CHUNK layers per test so that
# each test stays well inside its time limit.  Two layers run at once (the
# oracle releases the interpreter lock and spreads a layer's heads over
# threads).
@pytest.mark.parametrize("chunk", range(max(len(_chunks(synth.config(n).layers))
                                            for n in ("C3", "C5"))))
def test_full_size_every_layer_stage_parity(full, chunk):
    cfg, spec, out, cache = full["cfg"], full["spec"], full["out"], full["cache"]
    chunks = _chunks(spec.layers)
    if chunk >= len(chunks):
        pytest.skip(f"{full['name']} has {spec.layers} layers")
    layers = chunks[chunk]
    log(f"{full['name']}: stage parity on layers {layers[0]}-{layers[-1]}")

    def one(li):
        return check_block_stages(spec, cfg, cache, out, li, 0, check_scores=False,
                                  log=lambda m: None)

    with concurrent.futures.ThreadPoolExecutor(2) as ex:
        res = list(ex.map(one, layers))
    for li, r in zip(layers, res):
        log(f"  layer {li}: {r}")


@pytest.mark.parametrize("where", [0, 1, 2, 3])
def test_full_size_end_to_end_scores(full, where):
    # four layers spread over the depth (first, one third, two thirds, last)
    cfg, spec, out, cache = full["cfg"], full["spec"], full["out"], full["cache"]
    L = spec.layers
    li = [0, L // 3, (2 * L) // 3, L - 1][where]
    H, G, D, w = cfg.kv_heads, cfg.group, cfg.head_dim, cfg.window
    n = cache["cu_seqlens"][1]
    q = cache["q_win"][li, :w].double().cpu().numpy()
    k = cache["k"][li, :n].double().cpu().numpy()
    qpos = np.repeat(np.arange(n - w, n), G)
    scale = 1.0 / math.sqrt(D)

    def head(h):
        Q = q[:, h * G:(h + 1) * G].reshape(w * G, D)
        return oracle.scores(Q, qpos, np.ascontiguousarray(k[:, h]), scale)

    with concurrent.futures.ThreadPoolExecutor(H) as ex:
        refs = list(ex.map(head, range(H)))
    worst = 0.0
    for h in range(H):
        s_gpu = out["scores"][li, h, :n].numpy()
        r, sm = score_rel_err(s_gpu, refs[h])
        assert r <= 1e-4 and sm <= 1e-4, (li, h, r, sm)
        worst = max(worst, r)
    log(f"{full['name']} layer {li}: worst per-key mass error {worst:.2e}")


def test_full_size_decode_multi_item(full):
    """Decode of 32 new queries per sequence over the whole packed cache: the
    (unit, chunk) work list is longer than the persistent grid, so workgroups
    run several items each (LDS ring and accumulators reset between items)."""
    if full["name"] != "C3":
        pytest.skip("one full-size decode case (the 8B-shaped cache)")
    cfg, spec, bufs = full["cfg"], full["spec"], full["bufs"]
    tq = 32
    po = bufs.packed_offsets.cpu().numpy()
    rows = np.diff(po)
    items = int(np.sum((rows + DEC_KEYS - 1) // DEC_KEYS))
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    grid = cus * DEC_WG_PER_CU
    log(f"decode: {len(rows)} units, {items} work items, at most {grid} resident workgroups, "
        f"longest segment {rows.max()} rows")
    assert items > 1.5 * grid   # most workgroups run two or more items
    dev = torch.device("cuda:0")
    qn = synth.make_queries(cfg, tq, dev)
    out, lse = ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq,
                         with_lse=True, max_rows=int(rows.max()))
    torch.cuda.synchronize()
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    scale = 1.0 / math.sqrt(D)
    longest = int(np.argmax(rows))
    shortest = int(np.argmin(rows))
    rng = np.random.default_rng(11)
    sample = sorted({longest, shortest, *rng.choice(len(rows), 6, replace=False).tolist()})

    def one(u):
        li, h = divmod(u, H)
        seg = slice(int(po[u]), int(po[u + 1]))
        kp = bufs.k_packed[seg].double().cpu().numpy()
        vp = bufs.v_packed[seg].double().cpu().numpy()
        q = qn[li, :tq, h * G:(h + 1) * G].double().cpu().numpy().reshape(-1, D)
        ref, ref_lse = oracle.decode(q, kp, vp, scale)
        got = out[li, :tq, h * G:(h + 1) * G].cpu().numpy().reshape(-1, D)
        got_lse = lse[li, :tq, h * G:(h + 1) * G].cpu().numpy().reshape(-1)
        err = np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
        return float(err.max()), float(np.abs(got_lse - ref_lse).max())

    with concurrent.futures.ThreadPoolExecutor(len(sample)) as ex:
        res = list(ex.map(one, sample))
    for u, (e, dl) in zip(sample, res):
        log(f"  unit {u} ({rows[u]} rows): worst row error {e:.2e}, lse error {dl:.2e}")
        assert e <= 1e-4 and dl <= 1e-4, (u, e, dl)
