"""Parity at the real model widths and sequence lengths, on sampled outputs the oracle computes
one by one (through the C ABI, bf16, tolerance 2e-2):

* vision encode: one 1280-wide layer (16 heads of 80, MLP 5120) on two 1008x1008 images
  (5184 patches each) with the 2x2 merge to 3584 -- sampled merged tokens of both images; and a
  2-layer encoder with the same head size over 200 patches (a ragged last key tile) and over 288
  and 300 patches (a last query block of 32 and 44 queries), and over 1596 patches (keys cut into
  3 ranges merged by a second pass) -- every merged token;
* prefill: one 3584-wide GQA layer (28/4 heads of 128, SwiGLU 18944, vocab 152064) over
  1300 visual embeddings + 200 text tokens, and over a screenshot's 3354 + 225 -- last-row logits,
  greedy id, sampled K/V;
* decode: 4 and 20 sequences with ragged contexts of 1200..1500 tokens in a shuffled paged cache
  (random bf16 K/V shared with the oracle) -- logits of every sequence and the appended K/V; the
  small batch runs the step with its RMSNorms folded into the projections, the large one with
  separate residual + norm kernels; each on the whole GPU and on a 64-CU partition.
"""
import dataclasses

import numpy as np
import pytest

from oracle import vlm
from paper_2509_21301_amd import synth
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu

VIT1 = dataclasses.replace(synth.VIT_1008, layers=1)
LLM1 = dataclasses.replace(synth.LLM_28, layers=1)


def test_vit_layer_real_width(gpu_lib):
    import torch
    nova = gpu_lib
    w = synth.vit_weights(VIT1, seed=0)
    imgs = synth.image(2, VIT1.image_h, VIT1.image_w, seed=1)
    out = nova.Vit(VIT1, w).encode(torch.from_numpy(imgs).cuda().to(torch.bfloat16)).float().cpu().numpy()
    tokens = [0, 35, 36, 647, 1259, 1295]          # corners, row ends, the middle of the 36x36 grid
    for i in range(2):
        ref = vlm.vit_encode_tokens(imgs[i], w, VIT1, tokens)
        assert vlm.max_rel_err(out[i, tokens], ref) < sc.TOL_BF16, f"image {i}"


# 8 heads of 80 over a 10x20 patch grid: 200 keys leave a ragged last key tile (3 x 64 + 8) and
# the 256-query workgroup has two of its four waves idle and one half filled
VIT_D80 = synth.VitConfig(hidden=640, heads=8, mlp=1280, layers=2, patch=14, merge=2, out_hidden=256,
                          image_h=140, image_w=280, name="vit2_d80_ragged")


# The same encoder over 16x18 and 10x30 grids: 288 and 300 patches leave a last query block of 32
# and of 44 queries, which runs as a light block (one query group and one 32-key half of every tile
# per wave, halves merged at the end): with the second query group empty, and half filled.
VIT_D80_LIGHT32 = dataclasses.replace(VIT_D80, image_h=224, image_w=252, name="vit2_d80_light32")
VIT_D80_LIGHT44 = dataclasses.replace(VIT_D80, image_h=140, image_w=420, name="vit2_d80_light44")
# A 38x42 grid (1596 patches) on 2 images: 7 query blocks x 8 heads x 2 images = 112 workgroups
# fill a fifth of the GPU's slots, so the keys are cut into 3 ranges (9, 9 and 7 tiles of 64, the
# last one ragged: 1596 = 24 x 64 + 60) merged by a second pass; the last query block (60
# queries) is a light block.  The MLP hidden, which holds the ranges' partial rows, is 4x wide.
VIT_D80_KEYRANGES = dataclasses.replace(VIT_D80, mlp=2560, image_h=532, image_w=588, name="vit2_d80_keyranges")


@pytest.mark.parametrize("cfg", [VIT_D80, VIT_D80_LIGHT32, VIT_D80_LIGHT44, VIT_D80_KEYRANGES], ids=lambda c: c.name)
def test_vit_head80_ragged_keys(gpu_lib, cfg):
    import torch
    nova = gpu_lib
    w = synth.vit_weights(cfg, seed=4)
    imgs = synth.image(2, cfg.image_h, cfg.image_w, seed=6)
    out = nova.Vit(cfg, w).encode(torch.from_numpy(imgs).cuda().to(torch.bfloat16)).float().cpu().numpy()
    for i in range(2):
        ref = vlm.vit_encode(imgs[i], w, cfg)
        assert vlm.max_rel_err(out[i], ref) < sc.TOL_BF16, f"image {i}"


@pytest.fixture(scope="module")
def llm1():
    import torch
    from paper_2509_21301_amd import nova
    w = synth.llm_weights(LLM1, seed=0)
    return w, nova.Llm(LLM1, w)


# 1500 tokens (the benchmark's prompt) and 3579 (a 1092x2408 screenshot's 3354 visual tokens and 225
# text tokens, the serving prompt), whose MLP down projection runs as one unsplit 256x256 launch
@pytest.mark.parametrize("nv,nt", [(synth.LLM_VISION_TOKENS, synth.LLM_TEXT_TOKENS), (3354, 225)])
def test_prefill_layer_real_width(gpu_lib, llm1, nv, nt):
    import torch
    nova = gpu_lib
    w, llm = llm1
    vis = synth.vision_embeds(nv, LLM1.hidden)
    ids = synth.text_ids(nt, LLM1.vocab)
    s = nv + nt
    table, pool = synth.block_tables([s], LLM1.block, seed=5)
    kv = nova.KvPool(llm, pool)
    logits = torch.empty(LLM1.vocab, dtype=torch.float32, device="cuda")
    nxt = llm.prefill(torch.from_numpy(vis).cuda().to(torch.bfloat16), torch.from_numpy(ids).cuda(),
                      torch.from_numpy(table[0]).cuda(), kv, logits=logits)
    torch.cuda.synchronize()
    x = np.concatenate([vis, w["embed"][ids]], 0)
    rows = np.array(sorted({0, 777, nv - 1, nv, s - 80, s - 1}))
    hid, k, v = vlm.llm_layer_rows(x, w, 0, LLM1, rows)
    ref_logits = vlm.lm_head(hid[-1:], w, LLM1)[0]
    got = logits.cpu().numpy()
    assert vlm.max_rel_err(got, ref_logits) < sc.TOL_BF16
    top = np.sort(ref_logits)[::-1]
    if top[0] - top[1] > 2 * np.abs(got - ref_logits).max():
        assert int(nxt.item()) == int(np.argmax(ref_logits))
    k5 = kv.k5.float().cpu().numpy()
    v5 = kv.v5.float().cpu().numpy()
    for p in [0, 15, 16, 1000, s - 80, s - 1]:
        blk, slot = table[0][p // 16], p % 16
        assert vlm.max_rel_err(k5[0, blk, :, slot, :], k[p]) < sc.TOL_BF16
        assert vlm.max_rel_err(v5[0, blk, :, :, slot], v[p]) < sc.TOL_BF16


# the thin GEMMs split K by the stream's CU count: on a 64-CU partition the O and down
# projections run unsplit, the residual update and the folded norm in the direct epilogue.
# nan_tail: the cache slots after each sequence's new token (never written, never attended)
# hold NaN, which must not reach the outputs
@pytest.mark.parametrize("bsz,cus,nan_tail", [(4, None, False), (20, None, False), (4, 64, False), (20, 64, False),
                                              (20, None, True)])
def test_decode_real_width(gpu_lib, llm1, bsz, cus, nan_tail):
    import torch
    nova = gpu_lib
    w, llm = llm1
    cfg = LLM1
    ctx = [1500 - 15 * b for b in range(bsz)]                    # positions of the new tokens
    tables, pool = synth.block_tables([c + 1 for c in ctx], cfg.block, seed=9)
    rng = np.random.default_rng(3)
    kref = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    kref.k[:] = synth.bf16_round(rng.standard_normal(kref.k.shape, dtype=np.float32))
    kref.v[:] = synth.bf16_round(rng.standard_normal(kref.v.shape, dtype=np.float32))
    if nan_tail:
        for b, c in enumerate(ctx):
            kref.k[:, tables[b][c // cfg.block], :, c % cfg.block + 1:, :] = np.nan
            kref.v[:, tables[b][c // cfg.block], :, c % cfg.block + 1:, :] = np.nan
    kv = nova.KvPool(llm, pool)
    kv.k5.copy_(torch.from_numpy(kref.k.astype(np.float32)).to(torch.bfloat16))
    kv.v5.copy_(torch.from_numpy(np.swapaxes(kref.v, -1, -2).astype(np.float32)).to(torch.bfloat16))
    ids = synth.text_ids(bsz, cfg.vocab, seed=12)
    pos = np.array(ctx, np.int32)
    logits = torch.empty(bsz, cfg.vocab, dtype=torch.float32, device="cuda")
    stream = None if cus is None else nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(cus, 0))
    args = (torch.from_numpy(ids).cuda(), torch.from_numpy(pos).cuda(), torch.from_numpy(tables).cuda())
    torch.cuda.synchronize()
    nxt = llm.decode(*args, kv, max_ctx=max(ctx) + 1, logits=logits, stream=stream)
    torch.cuda.synchronize()
    ref_logits, ref_ids = vlm.llm_decode_step(ids, pos, tables, kref, w, cfg)
    got = logits.cpu().numpy()
    got_ids = nxt.cpu().numpy()
    for b in range(bsz):
        assert vlm.max_rel_err(got[b], ref_logits[b]) < sc.TOL_BF16, f"seq {b}"
        top = np.sort(ref_logits[b])[::-1]
        if top[0] - top[1] > 2 * np.abs(got[b] - ref_logits[b]).max():
            assert got_ids[b] == ref_ids[b], f"seq {b}"
    assert np.isfinite(got).all()
    gk, gv = kv.k5.float().cpu().numpy(), kv.v5.float().cpu().numpy()
    if nan_tail:   # the NaN slots must still be NaN on both sides (nothing wrote there), then compare the rest
        assert np.array_equal(np.isnan(gk), np.isnan(kref.k))
        assert np.array_equal(np.isnan(np.swapaxes(gv, -1, -2)), np.isnan(kref.v))
        kref.k, kref.v, gk, gv = (np.nan_to_num(a) for a in (kref.k, kref.v, gk, gv))
    ek, ev = sc.kv_errors(kref.k, kref.v, gk, gv)
    assert ek < sc.TOL_BF16 and ev < sc.TOL_BF16
