"""Oracle parity at the depths and shapes the benchmark runs, bf16, tolerance 2e-2 (no depth factor):

* vision encode through all 32 layers of the 1280-wide ViT on one 1008x1008 image (5184
  patches), sampled merged tokens (the oracle runs every layer on every patch, the last one at
  the sampled patches only);
* one 1280-wide encoder layer on a 1092x2408 screenshot (13,416 patches, a 78x172 grid, 3354
  merged tokens): the serving shape;
* the 3584-wide GQA decoder at 4 layers with the benchmark's 1500-token prompt (1300 visual + 200
  text): last-row logits and K/V of every layer, then one decode step at batch 1 continuing that
  prefill, and one at batch 32 over ragged 1300..1500-token contexts of random cached K/V;
* the same decoder at 8, 16 and its full 28 layers with a 256-token prompt: last-row logits, K/V
  of every layer and a batch-1 decode step continuing the prefill, and at 28 layers a batch-32
  step over random cached K/V.

Depth and bf16 storage.  A bf16 model keeps its activations and KV cache in bf16 between
operations, and every such store rounds by up to 2^-9 relative; the random decoder amplifies
these perturbations layer by layer.  Against the exact oracle the HIP path measures about 0.8%
at one decoder layer, 1.7% at 4, 2.0% at 8, 3.8% at 16 and 5.4% at 28, and the oracle itself
evaluated with its stores rounded to bf16 (oracle.vlm.bf16_store) moves away from the exact
oracle by the same order: the error at depth is what bf16 storage implies, not a defect of one
implementation.  So the decoder is held to 2e-2 against the exact oracle at 4 layers (the
benchmark's prompt), and at 8, 16 and 28 layers to the larger of 2e-2 and twice the distance
between the exact oracle and its bf16-storage evaluation, computed in the test for each output.
Each test prints the errors.

Weights are seeded draws on the device (torch's generator, bf16), copied to the host for the
oracle; both sides read the same values.
"""
import dataclasses

import numpy as np
import pytest

from oracle import vlm
from paper_2509_21301_amd import synth
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu

TOL = sc.TOL_BF16


def _report(name, **errs):
    print(f"[depth] {name}: " + ", ".join(f"{k} {v:.3e}" for k, v in errs.items()), flush=True)


# ------------------------------------------------------------------ vision encode
@pytest.mark.timeout(400)
def test_encode_32_layers_vs_oracle(gpu_lib):
    import torch
    nova = gpu_lib
    cfg = synth.VIT_1008
    wt = synth.vit_weights_torch(cfg, seed=3)
    vit = nova.Vit(cfg, wt)
    w = synth.to_host(wt)
    del wt
    img = synth.image(1, cfg.image_h, cfg.image_w, seed=7)
    out = vit.encode(torch.from_numpy(img).cuda().to(torch.bfloat16)).float().cpu().numpy()[0]
    tokens = [0, 17, 35, 36, 640, 647, 1000, 1259, 1295]      # corners, row ends, interior of the 36x36 grid
    ref = vlm.vit_encode_tokens(img[0], w, cfg, tokens)
    err = vlm.max_rel_err(out[tokens], ref)
    _report("encode ViT-32 1008x1008", merged_tokens=err)
    assert np.isfinite(out).all()
    assert err < TOL


@pytest.mark.timeout(300)
def test_encode_layer_screenshot_shape_vs_oracle(gpu_lib):
    import torch
    nova = gpu_lib
    cfg = dataclasses.replace(synth.VIT_SCREEN, layers=1)
    wt = synth.vit_weights_torch(cfg, seed=5)
    vit = nova.Vit(cfg, wt)
    w = synth.to_host(wt)
    del wt
    img = synth.image(1, cfg.image_h, cfg.image_w, seed=8)
    out = vit.encode(torch.from_numpy(img).cuda().to(torch.bfloat16)).float().cpu().numpy()[0]
    n_out, gw = cfg.n_out, cfg.grid_w // 2
    assert n_out == 3354 and gw == 86
    tokens = [0, gw - 1, gw, 1700, n_out - gw, n_out - 1]
    ref = vlm.vit_encode_tokens(img[0], w, cfg, tokens)
    err = vlm.max_rel_err(out[tokens], ref)
    _report("encode 1-layer 1092x2408", merged_tokens=err)
    assert err < TOL


# ------------------------------------------------------------------ LLM at depth
class _Model:
    """A seeded 3584-wide decoder on the device and its host copy for the oracle."""

    def __init__(self, nova, layers, seed):
        self.cfg = dataclasses.replace(synth.LLM_28, layers=layers)
        wt = synth.llm_weights_torch(self.cfg, seed=seed)
        self.llm = nova.Llm(self.cfg, wt)
        self.w = synth.to_host(wt)
        del wt


@pytest.fixture(scope="module")
def llm4(gpu_lib):
    m = _Model(gpu_lib, 4, seed=6)
    yield m
    del m


@pytest.fixture(scope="module")
def llm28(gpu_lib):
    m = _Model(gpu_lib, 28, seed=7)
    yield m
    del m


def _errors(got, ref):
    return vlm.max_rel_err(got, ref)


def _check_ids(got_logits, got_id, ref_logits, ref_id, what):
    top = np.sort(ref_logits)[::-1]
    if top[0] - top[1] > 2 * np.abs(got_logits - ref_logits).max():
        assert got_id == ref_id, what


def _prefill_then_decode(nova, m, nv, nt, name):
    """Prefill [nv visual ; nt text] on both sides, compare the last-row logits and every layer's
    K/V, then run one batch-1 decode step that feeds the exact oracle's greedy token at position
    S on each side's own cache.  Returns {output: (HIP path vs exact oracle, bf16-storage oracle
    vs exact oracle)}."""
    import torch
    cfg, w = m.cfg, m.w
    vis = synth.vision_embeds(nv, cfg.hidden, seed=11)
    ids = synth.text_ids(nt, cfg.vocab, seed=12)
    s = nv + nt
    table, pool = synth.block_tables([s + 1], cfg.block, seed=13)
    kv = nova.KvPool(m.llm, pool)
    logits = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    tab_d = torch.from_numpy(table).cuda()
    nxt = m.llm.prefill(torch.from_numpy(vis).cuda().to(torch.bfloat16), torch.from_numpy(ids).cuda(), tab_d[0], kv,
                        logits=logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    used = table[0][: (s + cfg.block - 1) // cfg.block]
    gk = kv.k5.float().cpu().numpy()[:, used]
    gv = np.swapaxes(kv.v5.float().cpu().numpy()[:, used], -1, -2)
    refs = {}
    for kind, store in (("exact", vlm._keep), ("bf16_store", vlm.bf16_store)):
        kref = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
        lg, tok = vlm.llm_prefill(vis, ids, w, cfg, kv=kref, table=table[0], store=store)
        refs[kind] = dict(logits=lg, tok=tok, kv=kref, k=kref.k[:, used].copy(), v=kref.v[:, used].copy())
    ex = refs["exact"]
    _check_ids(got, int(nxt.item()), ex["logits"], ex["tok"], "prefill id")
    feed = ex["tok"]                              # every side decodes the exact oracle's token
    dl = torch.empty(1, cfg.vocab, dtype=torch.float32, device="cuda")
    dn = m.llm.decode(torch.tensor([feed], dtype=torch.int32, device="cuda"),
                      torch.tensor([s], dtype=torch.int32, device="cuda"), tab_d, kv, max_ctx=s + 1, logits=dl)
    torch.cuda.synchronize()
    gdl, gdn = dl.cpu().numpy()[0], int(dn.item())
    for kind, store in (("exact", vlm._keep), ("bf16_store", vlm.bf16_store)):
        r = refs[kind]
        r["dl"] = vlm.llm_decode_step(np.array([feed]), np.array([s]), table, r["kv"], w, cfg, store=store)[0][0]
    _check_ids(gdl, gdn, ex["dl"], int(np.argmax(ex["dl"])), "decode id")
    st = refs["bf16_store"]
    k_err = lambda a, b: max(_errors(a[l], b[l]) for l in range(cfg.layers))
    out = {"prefill_logits": (_errors(got, ex["logits"]), _errors(st["logits"], ex["logits"])),
           "k": (k_err(gk, ex["k"]), k_err(st["k"], ex["k"])),
           "v": (k_err(gv, ex["v"]), k_err(st["v"], ex["v"])),
           "decode_b1_logits": (_errors(gdl, ex["dl"]), _errors(st["dl"], ex["dl"]))}
    _report(f"{name}: HIP path vs exact oracle", **{k: v[0] for k, v in out.items()})
    _report(f"{name}: bf16-storage oracle vs exact oracle", **{k: v[1] for k, v in out.items()})
    return out


def _decode_batch(nova, m, ctx, seed, name):
    """One decode step over len(ctx) sequences whose cached K/V are random bf16 values shared
    with the oracle (positions ctx[b], a shuffled paged cache).  Returns {output: (HIP path vs
    exact oracle, bf16-storage oracle vs exact oracle)}."""
    import torch
    cfg, w = m.cfg, m.w
    bsz = len(ctx)
    tables, pool = synth.block_tables([c + 1 for c in ctx], cfg.block, seed=seed)
    rng = np.random.default_rng(seed)
    k0 = synth.bf16_round(rng.standard_normal((cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim), dtype=np.float32))
    v0 = synth.bf16_round(rng.standard_normal((cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim), dtype=np.float32))
    kv = nova.KvPool(m.llm, pool)
    kv.k5.copy_(torch.from_numpy(k0).to(torch.bfloat16))
    kv.v5.copy_(torch.from_numpy(np.ascontiguousarray(np.swapaxes(v0, -1, -2))).to(torch.bfloat16))
    ids = synth.text_ids(bsz, cfg.vocab, seed=seed + 1)
    pos = np.array(ctx, np.int32)
    logits = torch.empty(bsz, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = m.llm.decode(torch.from_numpy(ids).cuda(), torch.from_numpy(pos).cuda(), torch.from_numpy(tables).cuda(), kv,
                       max_ctx=max(ctx) + 1, logits=logits)
    torch.cuda.synchronize()
    got, got_ids = logits.cpu().numpy(), nxt.cpu().numpy()
    gk, gv = kv.k5.float().cpu().numpy(), np.swapaxes(kv.v5.float().cpu().numpy(), -1, -2)
    refs = {}
    for kind, store in (("exact", vlm._keep), ("bf16_store", vlm.bf16_store)):
        kref = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
        kref.k[:] = k0
        kref.v[:] = v0
        lg, nid = vlm.llm_decode_step(ids, pos, tables, kref, w, cfg, store=store)
        refs[kind] = dict(logits=lg, ids=nid, k=kref.k, v=kref.v)
    ex, st = refs["exact"], refs["bf16_store"]
    for b in range(bsz):
        _check_ids(got[b], int(got_ids[b]), ex["logits"][b], int(ex["ids"][b]), f"seq {b}")
    per_seq = lambda a: max(_errors(a[b], ex["logits"][b]) for b in range(bsz))
    out = {"decode_logits": (per_seq(got), per_seq(st["logits"])),
           "k": (_errors(gk, ex["k"]), _errors(st["k"], ex["k"])),
           "v": (_errors(gv, ex["v"]), _errors(st["v"], ex["v"]))}
    _report(f"{name}: HIP path vs exact oracle", **{k: v[0] for k, v in out.items()})
    _report(f"{name}: bf16-storage oracle vs exact oracle", **{k: v[1] for k, v in out.items()})
    return out


def _beyond_exact_bound(errs):
    """Outputs whose error against the exact oracle reaches 2e-2."""
    return {k: v[0] for k, v in errs.items() if v[0] >= TOL}


def _beyond_depth_bound(errs):
    """Outputs whose error against the exact oracle reaches max(2e-2, twice the bf16-storage
    oracle's own distance from the exact one)."""
    return {k: v for k, v in errs.items() if v[0] >= max(TOL, 2.0 * v[1])}


@pytest.mark.timeout(400)
def test_llm4_prefill_1500_then_decode_vs_oracle(gpu_lib, llm4):
    errs = _prefill_then_decode(gpu_lib, llm4, synth.LLM_VISION_TOKENS, synth.LLM_TEXT_TOKENS, "LLM 4x3584 S=1500")
    assert not _beyond_exact_bound(errs)


@pytest.mark.timeout(400)
def test_llm4_decode_batch32_vs_oracle(gpu_lib, llm4):
    ctx = [1500 - 6 * b for b in range(32)]
    errs = _decode_batch(gpu_lib, llm4, ctx, seed=21, name="LLM 4x3584 decode B=32")
    assert not _beyond_exact_bound(errs)


@pytest.mark.timeout(400)
@pytest.mark.parametrize("layers", [8, 16])
def test_llm_depth_prefill_then_decode_vs_oracle(gpu_lib, layers):
    m = _Model(gpu_lib, layers, seed=7)
    errs = _prefill_then_decode(gpu_lib, m, 200, 56, f"LLM {layers}x3584 S=256")
    assert not _beyond_depth_bound(errs)


@pytest.mark.timeout(400)
def test_llm28_prefill_then_decode_vs_oracle(gpu_lib, llm28):
    errs = _prefill_then_decode(gpu_lib, llm28, 200, 56, "LLM 28x3584 S=256")
    assert not _beyond_depth_bound(errs)


@pytest.mark.timeout(400)
def test_llm28_decode_batch32_vs_oracle(gpu_lib, llm28):
    ctx = [256 - 3 * b for b in range(32)]
    errs = _decode_batch(gpu_lib, llm28, ctx, seed=31, name="LLM 28x3584 decode B=32")
    assert not _beyond_depth_bound(errs)
