"""Batched paged decode and ragged prefill against the oracle (tiny LLM, through the C ABI).

20 sequences (more than one 16-wide MFMA column group) with ragged prompt lengths, some with
no visual tokens and one with no text, share a shuffled block pool; two in-flight decode steps
run on the whole batch."""
import numpy as np
import pytest

from oracle import vlm
from paper_2509_21301_amd import synth
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu

LENS = [(0, 5), (3, 1), (17, 0), (31, 2), (16, 16), (40, 9), (1, 63), (64, 1), (0, 77), (12, 12),
        (50, 30), (7, 7), (33, 1), (2, 2), (45, 0), (0, 16), (29, 35), (9, 40), (15, 1), (60, 4)]
STEPS = 2


def _inputs():
    cfg = synth.TINY_LLM
    w = synth.llm_weights(cfg, 0)
    vis = [synth.vision_embeds(nv, cfg.hidden, seed=100 + i) if nv else np.zeros((0, cfg.hidden), np.float32)
           for i, (nv, _) in enumerate(LENS)]
    ids = [synth.text_ids(nt, cfg.vocab, seed=200 + i) if nt else np.zeros(0, np.int32)
           for i, (_, nt) in enumerate(LENS)]
    lens = [nv + nt for nv, nt in LENS]
    tables, pool = synth.block_tables([n + STEPS for n in lens], cfg.block, seed=11)
    return cfg, w, vis, ids, lens, tables, pool


@pytest.fixture(scope="module")
def ref():
    cfg, w, vis, ids, lens, tables, pool = _inputs()
    kv = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    pre = [vlm.llm_prefill(vis[b], ids[b], w, cfg, kv=kv, table=tables[b]) for b in range(len(LENS))]
    toks = np.array([t for _, t in pre], np.int32)
    steps = []
    feed = toks
    for t in range(STEPS):
        lg, nx = vlm.llm_decode_step(feed, np.array(lens) + t, tables, kv, w, cfg)
        steps.append((feed.copy(), lg, nx))
        feed = nx
    return dict(cfg=cfg, w=w, vis=vis, ids=ids, lens=lens, tables=tables, pool=pool, pre=pre, steps=steps, kv=kv)


def _gpu(nova, act, ref):
    import torch
    cfg, dev = ref["cfg"], "cuda"
    llm = nova.Llm(cfg, ref["w"], act=act)
    kv = nova.KvPool(llm, ref["pool"])
    tables = torch.from_numpy(ref["tables"]).to(dev)
    dt = nova.act_dtype(act)
    pre_logits, pre_tok = [], []
    for b in range(len(LENS)):
        vis = torch.from_numpy(ref["vis"][b]).to(dev, dt) if LENS[b][0] else None
        ids = torch.from_numpy(ref["ids"][b]).to(dev) if LENS[b][1] else torch.zeros(0, dtype=torch.int32, device=dev)
        lg = torch.empty(cfg.vocab, dtype=torch.float32, device=dev)
        nx = llm.prefill(vis, ids, tables[b], kv, logits=lg)
        pre_logits.append(lg.cpu().numpy())
        pre_tok.append(int(nx.item()))
    steps = []
    lens = np.array(ref["lens"])
    for t in range(STEPS):
        feed = torch.from_numpy(ref["steps"][t][0]).to(dev)      # teacher-forced on the oracle's ids
        pos = torch.from_numpy((lens + t).astype(np.int32)).to(dev)
        lg = torch.empty(len(LENS), cfg.vocab, dtype=torch.float32, device=dev)
        nx = llm.decode(feed, pos, tables, kv, max_ctx=int(lens.max()) + STEPS, logits=lg)
        torch.cuda.synchronize()
        steps.append((lg.cpu().numpy(), nx.cpu().numpy()))
    return pre_logits, pre_tok, steps, kv


@pytest.mark.parametrize("mode", ["f32", "bf16"])
def test_ragged_prefill_and_batched_decode(gpu_lib, ref, mode):
    act = gpu_lib.ACT_F32 if mode == "f32" else gpu_lib.ACT_BF16
    tol = sc.TOL_F32 if mode == "f32" else sc.TOL_BF16
    pre_logits, pre_tok, steps, kv = _gpu(gpu_lib, act, ref)
    for b, (lg, tok) in enumerate(ref["pre"]):
        assert vlm.max_rel_err(pre_logits[b], lg) < tol, f"prefill seq {b}"
        if mode == "f32":
            assert pre_tok[b] == tok, f"prefill seq {b}"
    for t, ((_, lg_ref, nx_ref), (lg, nx)) in enumerate(zip(ref["steps"], steps)):
        for b in range(len(LENS)):
            assert vlm.max_rel_err(lg[b], lg_ref[b]) < tol, f"step {t} seq {b}"
        if mode == "f32":
            assert np.array_equal(nx, nx_ref), f"step {t}"
    ek, ev = sc.kv_errors(ref["kv"].k, ref["kv"].v, kv.k5.float().cpu().numpy(), kv.v5.float().cpu().numpy())
    assert ek < tol and ev < tol


def test_long_prefill_every_position(gpu_lib):
    """A 700-token bf16 prefill (600 visual + 100 text) on the tiny LLM: six causal query blocks
    of 128 (2 .. 11 key tiles of 64, the last block ragged).  Last-row logits and the K/V of both
    layers at every position (layer 1's K/V come from layer 0's attention output of every row)
    against the oracle."""
    import torch
    nova = gpu_lib
    cfg = synth.TINY_LLM
    w = synth.llm_weights(cfg, 0)
    nv, nt = 600, 100
    vis = synth.vision_embeds(nv, cfg.hidden, seed=31)
    ids = synth.text_ids(nt, cfg.vocab, seed=32)
    tables, pool = synth.block_tables([nv + nt], cfg.block, seed=33)
    kv_ref = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    lg_ref, _ = vlm.llm_prefill(vis, ids, w, cfg, kv=kv_ref, table=tables[0])
    llm = nova.Llm(cfg, w, act=nova.ACT_BF16)
    kv = nova.KvPool(llm, pool)
    lg = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    llm.prefill(torch.from_numpy(vis).to("cuda", torch.bfloat16), torch.from_numpy(ids).to("cuda"),
                torch.from_numpy(tables[0]).to("cuda"), kv, logits=lg)
    torch.cuda.synchronize()
    assert vlm.max_rel_err(lg.cpu().numpy(), lg_ref) < sc.TOL_BF16
    ek, ev = sc.kv_errors(kv_ref.k, kv_ref.v, kv.k5.float().cpu().numpy(), kv.v5.float().cpu().numpy())
    assert ek < sc.TOL_BF16 and ev < sc.TOL_BF16, (ek, ev)
