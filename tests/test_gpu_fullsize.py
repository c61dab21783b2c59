"""The stages at the sizes and launch configurations bench.py times, checked through properties
that hold at any size (the oracle would need minutes per image or sequence at full depth; the
real-width single-layer tests hold the kernels to the oracle at these shapes):

* vision encode, ViT-32 (1280 wide, 32 layers) on 8 images of 1008x1008 in one batch: a second
  pass repeats the first bit for bit, every value is finite, and each image's output matches its
  output when encoded alone -- rows never mix, but the one-image pass is a different bf16 path: its
  attention cuts the keys into 3 ranges merged from bf16 partial rows (one image's query blocks
  fill a third of the workgroup slots less), so the two agree within the two-path depth bound;
* prefill of 1300 visual + 200 text tokens through the 28-layer 3584-wide LLM, against a
  prefill of the first 1499 tokens followed by one decode step on the 1500th: the same last-row
  logits through other kernels (GEMM and tiled attention against thin GEMM and paged decode
  attention), and the same K/V for the shared prefix;
* decode at batch 32 with contexts of 1564 tokens (the unfused path) against batch 8 (the path
  with the RMSNorms folded into the projections) and batch 1 on the same sequences.
Weights are random, as in the benchmark (seeded N(0, 0.02) bf16, unit norm gains).

Tolerance between two bf16 paths at full depth: at one layer both sit within the 2e-2 of the
oracle; the two paths round in different orders at every layer, and independent per-layer
rounding grows like the square root of the depth, so the bound is 2e-2 * sqrt(L) (measured: 0.8%
at one layer, 1.8% at 8, 3.7% at 28 for prefill against prefix + decode).  Computations that are
the same row by row (a prefix of the prompt) must agree exactly.
"""
import math

import numpy as np
import pytest

import bench
from oracle import vlm
from paper_2509_21301_amd import synth
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu


def depth_tol(layers):
    return sc.TOL_BF16 * math.sqrt(layers)


def test_encode_bench_config_batch_invariant(gpu_lib):
    import torch
    nova = gpu_lib
    cfg = synth.VIT_1008
    vit = bench.build_vit(nova, cfg, "cuda")
    px = torch.from_numpy(synth.image(8, cfg.image_h, cfg.image_w, seed=1)).to("cuda", torch.bfloat16).contiguous()
    out = vit.encode(px)
    again = vit.encode(px)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert torch.equal(out, again)
    for i in (0, 5, 7):
        alone = vit.encode(px[i:i + 1].contiguous())
        err = vlm.max_rel_err(alone[0].float().cpu().numpy(), out[i].float().cpu().numpy())
        print(f"image {i} alone vs in the batch: max rel err {err:.2e}")
        assert err < depth_tol(cfg.layers), f"image {i}: {err}"


@pytest.fixture(scope="module")
def llm28(gpu_lib):
    return bench.build_llm(gpu_lib, synth.LLM_28, "cuda")


def test_prefill_matches_prefix_plus_decode_step(gpu_lib, llm28):
    import torch
    nova = gpu_lib
    cfg = synth.LLM_28
    nv, nt = synth.LLM_VISION_TOKENS, synth.LLM_TEXT_TOKENS
    s = nv + nt
    vis = torch.from_numpy(synth.vision_embeds(nv, cfg.hidden)).to("cuda", torch.bfloat16)
    ids = torch.from_numpy(synth.text_ids(nt, cfg.vocab)).to("cuda")
    tables, pool = synth.block_tables([s, s], cfg.block, seed=5)
    kv = nova.KvPool(llm28, pool)
    tab = torch.from_numpy(tables).to("cuda")
    full = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    nxt_full = llm28.prefill(vis, ids, tab[0], kv, logits=full)
    # the same prompt without its last token, in the second sequence's blocks, then one decode step
    llm28.prefill(vis, ids[:-1], tab[1], kv)
    step = torch.empty(1, cfg.vocab, dtype=torch.float32, device="cuda")
    pos = torch.tensor([s - 1], dtype=torch.int32, device="cuda")
    nxt_step = llm28.decode(ids[-1:].contiguous(), pos, tab[1:2].contiguous(), kv, max_ctx=s, logits=step)
    torch.cuda.synchronize()
    a, b = full.cpu().numpy(), step[0].cpu().numpy()
    assert np.isfinite(a).all() and vlm.max_rel_err(b, a) < depth_tol(cfg.layers)
    top = np.sort(a)[::-1]
    if top[0] - top[1] > 2 * np.abs(a - b).max():
        assert int(nxt_full.item()) == int(nxt_step.item())
    # K/V of the shared prefix, every layer: causal rows computed the same way, so equal bit for
    # bit; the last token's, written by the decode step, within the depth bound
    k5, v5 = kv.k5, kv.v5
    for p in (0, 15, 16, 777, nv - 1, nv, s - 2):
        b0, b1, sl = tables[0][p // cfg.block], tables[1][p // cfg.block], p % cfg.block
        assert torch.equal(k5[:, b0, :, sl, :], k5[:, b1, :, sl, :]), f"K, position {p}"
        assert torch.equal(v5[:, b0, :, :, sl], v5[:, b1, :, :, sl]), f"V, position {p}"
    b0, b1, sl = tables[0][(s - 1) // cfg.block], tables[1][(s - 1) // cfg.block], (s - 1) % cfg.block
    for l in range(cfg.layers):
        tol = depth_tol(l + 1)
        ka, kb = k5[l, b0, :, sl, :].float().cpu().numpy(), k5[l, b1, :, sl, :].float().cpu().numpy()
        va, vb = v5[l, b0, :, :, sl].float().cpu().numpy(), v5[l, b1, :, :, sl].float().cpu().numpy()
        assert vlm.max_rel_err(kb, ka) < tol and vlm.max_rel_err(vb, va) < tol, f"last token, layer {l}"


def test_decode_bench_config_batches_agree(gpu_lib, llm28):
    import torch
    nova = gpu_lib
    cfg = synth.LLM_28
    ctx_max = synth.LLM_VISION_TOKENS + synth.LLM_TEXT_TOKENS + synth.LLM_DECODE_STEPS
    tables, pool = synth.block_tables([ctx_max] * 32, cfg.block, seed=5)
    kv = nova.KvPool(llm28, pool)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    kv.k.copy_((torch.randn(kv.k.numel(), generator=g, device="cuda") * 0.5).to(kv.k.dtype))
    kv.v.copy_((torch.randn(kv.v.numel(), generator=g, device="cuda") * 0.5).to(kv.v.dtype))
    tab = torch.from_numpy(tables).to("cuda")
    ids = torch.from_numpy(synth.text_ids(32, cfg.vocab, seed=9)).to("cuda")
    # ragged positions up to the benchmark's last one; each step writes only its own position
    pos = torch.tensor([ctx_max - 1 - 3 * b for b in range(32)], dtype=torch.int32, device="cuda")

    def step(sel):
        lg = torch.empty(len(sel), cfg.vocab, dtype=torch.float32, device="cuda")
        nx = llm28.decode(ids[sel].contiguous(), pos[sel].contiguous(), tab[sel].contiguous(), kv, ctx_max, logits=lg)
        torch.cuda.synchronize()
        return lg.cpu().numpy(), nx.cpu().numpy()

    lg32, nx32 = step(list(range(32)))
    assert np.isfinite(lg32).all()
    lg8, nx8 = step(list(range(8)))
    lg1, nx1 = step([31])
    for got, ref_row, gid, rid, what in [(lg8[b], lg32[b], nx8[b], nx32[b], f"seq {b}, batch 8") for b in range(8)] + \
                                         [(lg1[0], lg32[31], nx1[0], nx32[31], "seq 31, batch 1")]:
        assert vlm.max_rel_err(got, ref_row) < depth_tol(cfg.layers), what
        top = np.sort(ref_row)[::-1]
        if top[0] - top[1] > 2 * np.abs(got - ref_row).max():
            assert gid == rid, what
