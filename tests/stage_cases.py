"""Shared drivers for the stage parity tests: run the tiny VLM stack through the oracle and
through libnova on the same seeded inputs (imported by the GPU tests and by smoke())."""
from __future__ import annotations

import numpy as np

from oracle import vlm
from paper_2509_21301_amd import synth

TOL_BF16 = 2e-2       # max relative error for bf16 activations
TOL_F32 = 2e-4        # fp32 exact mode: bf16 hi+lo operands, fp32 accumulation


def oracle_tiny(decode_steps=synth.TINY_DECODE_STEPS, n_text=synth.TINY_TEXT, forced=None):
    """Oracle run of the tiny stack: encode -> prefill -> greedy decode (or decode fed ``forced``)."""
    vc, lc = synth.TINY_VIT, synth.TINY_LLM
    wv, wl = synth.vit_weights(vc, 0), synth.llm_weights(lc, 0)
    img = synth.image(1, vc.image_h, vc.image_w, seed=1)
    ids = synth.text_ids(n_text, lc.vocab, seed=2)
    vis = vlm.vit_encode(img[0], wv, vc)
    s = vis.shape[0] + n_text
    table, pool = synth.block_tables([s + decode_steps], lc.block, seed=5)
    kv = vlm.PagedKV(lc.layers, pool, lc.n_kv, lc.block, lc.head_dim)
    logits0, tok = vlm.llm_prefill(vis, ids, wl, lc, kv=kv, table=table[0])
    kv_after_prefill = (kv.k.copy(), kv.v.copy())
    toks, logs = [tok], [logits0]
    for t in range(decode_steps):
        feed = toks[-1] if forced is None else forced[t]
        lg, nx = vlm.llm_decode_step(np.array([feed]), np.array([s + t]), table, kv, wl, lc)
        logs.append(lg[0])
        toks.append(int(nx[0]))
    return dict(img=img, ids=ids, vis=vis, table=table, pool=pool, logits=logs, tokens=toks, kv=kv,
                kv_prefill=kv_after_prefill, wv=wv, wl=wl, s=s)


def gpu_tiny(nova, act, ref, decode_steps=synth.TINY_DECODE_STEPS, forced=None):
    """The same run through libnova on cuda:0; returns host copies of every stage output."""
    import torch
    vc, lc = synth.TINY_VIT, synth.TINY_LLM
    dev = "cuda"
    vit = nova.Vit(vc, ref["wv"], act=act)
    llm = nova.Llm(lc, ref["wl"], act=act)
    pixels = torch.from_numpy(ref["img"]).to(dev, torch.bfloat16).contiguous()
    vis = vit.encode(pixels)[0]
    ids = torch.from_numpy(ref["ids"]).to(dev)
    table = torch.from_numpy(ref["table"]).to(dev)
    kv = nova.KvPool(llm, ref["pool"])
    logits = torch.empty(lc.vocab, dtype=torch.float32, device=dev)
    nxt = llm.prefill(vis, ids, table[0], kv, logits=logits)
    torch.cuda.synchronize()
    out = dict(vis=vis.float().cpu().numpy(), logits=[logits.cpu().numpy()], tokens=[int(nxt.item())],
               k_prefill=kv.k5.float().cpu().numpy(), v_prefill=kv.v5.float().cpu().numpy())
    s = ref["s"]
    tok = nxt
    lg = torch.empty(1, lc.vocab, dtype=torch.float32, device=dev)
    for t in range(decode_steps):
        feed = tok if forced is None else torch.tensor([forced[t]], dtype=torch.int32, device=dev)
        pos = torch.tensor([s + t], dtype=torch.int32, device=dev)
        tok = llm.decode(feed, pos, table, kv, max_ctx=s + decode_steps, logits=lg)
        torch.cuda.synchronize()
        out["logits"].append(lg[0].cpu().numpy())
        out["tokens"].append(int(tok.item()))
    out["k_final"] = kv.k5.float().cpu().numpy()
    out["v_final"] = kv.v5.float().cpu().numpy()
    return out


def kv_errors(ref_k, ref_v, gpu_k5, gpu_v5):
    """Relative errors of the paged cache: GPU V blocks are stored [d][slot]."""
    return vlm.max_rel_err(gpu_k5, ref_k), vlm.max_rel_err(np.swapaxes(gpu_v5, -1, -2), ref_v)
