"""The allocation-free decode entry point (nova_llm_decode_noalloc) against nova_llm_decode, through
the C ABI: on the same inputs the two run the same kernels, so next ids, logits and the appended
K/V must agree bit for bit.  Two calls in a row, the second with a smaller batch and shorter
contexts (the static scratch keeps the first call's contents), on the tiny stack in both
activation modes and on one 3584-wide layer; and a step whose workspace exceeds the scratch is
refused before anything is launched."""
import dataclasses

import numpy as np
import pytest

from paper_2509_21301_amd import synth

pytestmark = pytest.mark.gpu


def _random_cache(nova, llm, cfg, pool, seed):
    import torch
    kv = nova.KvPool(llm, pool)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    kv.k.copy_(torch.randn(kv.k.numel(), generator=g, device="cuda").to(kv.k.dtype))
    kv.v.copy_(torch.randn(kv.v.numel(), generator=g, device="cuda").to(kv.v.dtype))
    return kv


def _clone_cache(nova, llm, pool, src):
    kv = nova.KvPool(llm, pool)
    kv.k.copy_(src.k)
    kv.v.copy_(src.v)
    return kv


def _compare(nova, llm, cfg, ctxs, seed):
    import torch
    dt = torch.float32
    for i, ctx in enumerate(ctxs):
        bsz = len(ctx)
        tables, pool = synth.block_tables([c + 1 for c in ctx], cfg.block, seed=seed + i)
        kv_a = _random_cache(nova, llm, cfg, pool, seed + 10 * i)
        kv_b = _clone_cache(nova, llm, pool, kv_a)
        ids = torch.from_numpy(synth.text_ids(bsz, cfg.vocab, seed=seed + i)).cuda()
        pos = torch.tensor(ctx, dtype=torch.int32, device="cuda")
        tab = torch.from_numpy(tables).cuda()
        la = torch.full((bsz, cfg.vocab), np.nan, dtype=dt, device="cuda")
        lb = torch.full((bsz, cfg.vocab), np.nan, dtype=dt, device="cuda")
        na = torch.full((bsz,), -1, dtype=torch.int32, device="cuda")
        nb = torch.full((bsz,), -1, dtype=torch.int32, device="cuda")
        max_ctx = max(ctx) + 1
        llm.decode(ids, pos, tab, kv_a, max_ctx, next_ids=na, logits=la)
        llm.decode_noalloc(ids, pos, tab, kv_b, max_ctx, next_ids=nb, logits=lb)
        torch.cuda.synchronize()
        assert torch.isfinite(la).all(), f"call {i}"
        assert torch.equal(na, nb), f"call {i}: next ids differ"
        assert torch.equal(la, lb), f"call {i}: logits differ"
        assert torch.equal(kv_a.k, kv_b.k) and torch.equal(kv_a.v, kv_b.v), f"call {i}: appended K/V differ"


@pytest.mark.parametrize("act", ["bf16", "f32"])
def test_noalloc_decode_tiny(gpu_lib, act):
    nova = gpu_lib
    cfg = synth.TINY_LLM
    llm = nova.Llm(cfg, synth.llm_weights(cfg, seed=0), act=nova.ACT_BF16 if act == "bf16" else nova.ACT_F32)
    # 12 sequences up to 200 tokens, then 3 sequences up to 40 tokens
    _compare(nova, llm, cfg, [[200 - 13 * b for b in range(12)], [40, 17, 33]], seed=40)


def test_noalloc_decode_real_width(gpu_lib):
    nova = gpu_lib
    cfg = dataclasses.replace(synth.LLM_28, layers=1)
    llm = nova.Llm(cfg, synth.llm_weights_torch(cfg, seed=2))
    # 20 sequences of 1200..1500 tokens (the unfused large-batch path), then 4 of 600..700 (folded)
    _compare(nova, llm, cfg, [[1500 - 15 * b for b in range(20)], [700, 655, 610, 601]], seed=50)


def test_noalloc_rejects_a_step_beyond_the_scratch(gpu_lib):
    import torch
    nova = gpu_lib
    # a 256-wide layer with a 600k-wide MLP: its batch-32 hidden activations alone take 38 MB
    cfg = dataclasses.replace(synth.TINY_LLM, inter=600_000, layers=1)
    (lo, lb), (ho, hb) = nova.llm_layouts(cfg)
    blobs = (torch.zeros(cfg.vocab, cfg.hidden, dtype=torch.bfloat16, device="cuda"),
             torch.zeros(lb // 2, dtype=torch.bfloat16, device="cuda"),
             torch.zeros(hb // 2, dtype=torch.bfloat16, device="cuda"), lb)
    llm = nova.Llm(cfg, None, blobs=blobs)
    assert nova.lib.nova_llm_decode_workspace_bytes(llm.h, 32, 64) > (32 << 20)
    tables, pool = synth.block_tables([64] * 32, cfg.block, seed=3)
    kv = nova.KvPool(llm, pool)
    ids = torch.zeros(32, dtype=torch.int32, device="cuda")
    pos = torch.full((32,), 63, dtype=torch.int32, device="cuda")
    nxt = torch.full((32,), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(nova.NovaError) as e:
        llm.decode_noalloc(ids, pos, torch.from_numpy(tables).cuda(), kv, 64, next_ids=nxt)
    assert e.value.code == nova.ENOSPACE and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (nxt == -7).all()                     # nothing ran
