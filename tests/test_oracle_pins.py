"""Pins for the oracle: each test ties an oracle function to something other than itself --
an independent library implementation, a closed form, an invariant, or a value the paper
prints -- so that a dropped term, a wrong sign or index, or a transposed operand fails."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import sched, vlm
from paper_2509_21301_amd import synth

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
RNG = np.random.default_rng(1234)


def t64(a):
    return torch.from_numpy(np.asarray(a, np.float64))


# ----------------------------------------------------------------------------- elementwise
def test_softmax_rows_sum_to_one_and_mask_zero():
    s = RNG.standard_normal((7, 13)) * 5
    s[:, 3] = -np.inf
    p = vlm.softmax(s)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-12)
    assert np.all(p[:, 3] == 0.0)
    assert np.allclose(p, torch.softmax(t64(s), -1).numpy(), atol=1e-14)


def test_norms_and_activations_match_torch():
    x = RNG.standard_normal((5, 48)) * 3 + 1
    g = RNG.standard_normal(48)
    b = RNG.standard_normal(48)
    assert np.allclose(vlm.layer_norm(x, g, b, 1e-6),
                       F.layer_norm(t64(x), (48,), t64(g), t64(b), eps=1e-6).numpy(), atol=1e-12)
    assert np.allclose(vlm.rms_norm(x, g, 1e-6), F.rms_norm(t64(x), (48,), t64(g), eps=1e-6).numpy(), atol=1e-12)
    assert np.allclose(vlm.gelu(x), F.gelu(t64(x)).numpy(), atol=1e-14)
    assert np.allclose(vlm.silu(x), F.silu(t64(x)).numpy(), atol=1e-14)


def test_norm_statistics():
    x = RNG.standard_normal((4, 64)) * 7 - 2
    y = vlm.layer_norm(x, np.ones(64), np.zeros(64), 0.0)
    assert np.allclose(y.mean(-1), 0, atol=1e-12) and np.allclose(y.var(-1), 1, atol=1e-12)
    r = vlm.rms_norm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt((r * r).mean(-1)), 1, atol=1e-12)


# ----------------------------------------------------------------------------- attention
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("nq,nkv", [(4, 4), (4, 2), (6, 1)])
def test_attention_matches_torch_sdpa(causal, nq, nkv):
    s, d = 11, 8
    q = RNG.standard_normal((s, nq, d))
    k = RNG.standard_normal((s, nkv, d))
    v = RNG.standard_normal((s, nkv, d))
    pos = np.arange(s)
    ours = vlm.attention(q, k, v, causal=causal, q_pos=pos, k_pos=pos)
    ref = F.scaled_dot_product_attention(t64(q).permute(1, 0, 2)[None], t64(k).permute(1, 0, 2)[None],
                                         t64(v).permute(1, 0, 2)[None], is_causal=causal,
                                         enable_gqa=(nq != nkv))[0].permute(1, 0, 2).numpy()
    assert np.allclose(ours, ref, atol=1e-12)


def test_attention_closed_forms():
    s, d = 9, 4
    v = RNG.standard_normal((s, 1, d))
    k = RNG.standard_normal((s, 1, d))
    # zero query: uniform weights -> mean of the values
    out = vlm.attention(np.zeros((3, 1, d)), k, v)
    assert np.allclose(out, v[:, 0].mean(0)[None, None], atol=1e-14)
    # causal, query 0 sees only key 0
    pos = np.arange(s)
    out = vlm.attention(RNG.standard_normal((s, 1, d)), k, v, causal=True, q_pos=pos, k_pos=pos)
    assert np.allclose(out[0, 0], v[0, 0], atol=1e-14)
    # one dominant key
    k2 = np.zeros((s, 1, d))
    k2[5, 0, 0] = 100.0
    out = vlm.attention(np.ones((1, 1, d)) * 10, k2, v)
    assert np.allclose(out[0, 0], v[5, 0], atol=1e-12)


def test_causal_rows_ignore_future_tokens_bit_exact():
    s, d = 12, 8
    q, k, v = (RNG.standard_normal((s, 2, d)) for _ in range(3))
    pos = np.arange(s)
    a = vlm.attention(q, k, v, causal=True, q_pos=pos, k_pos=pos)
    k2, v2 = k.copy(), v.copy()
    k2[7:] += 3.0
    v2[7:] -= 5.0
    b = vlm.attention(q, k2, v2, causal=True, q_pos=pos, k_pos=pos)
    assert np.array_equal(a[:7], b[:7])
    assert not np.allclose(a[7:], b[7:])


def test_gqa_equals_mha_with_replicated_kv():
    s, d = 10, 8
    q = RNG.standard_normal((s, 6, d))
    k = RNG.standard_normal((s, 2, d))
    v = RNG.standard_normal((s, 2, d))
    pos = np.arange(s)
    a = vlm.attention(q, k, v, causal=True, q_pos=pos, k_pos=pos)
    b = vlm.attention(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), causal=True, q_pos=pos, k_pos=pos)
    assert np.array_equal(a, b)


# ----------------------------------------------------------------------------- rope
def test_rope_worked_example_half_split():
    # d = 4: dims (0,2) rotate at frequency 1, dims (1,3) at theta^-1/2.
    x = np.array([[[1.0, 0.0, 0.0, 0.0]]])
    y = vlm.rope(x, np.array([1]), 10000.0)
    assert np.allclose(y[0, 0], [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    y = vlm.rope(x, np.array([3]), 10000.0)
    a = 3 * 10000.0 ** -0.5
    assert np.allclose(y[0, 0], [0, math.cos(a), 0, math.sin(a)], atol=1e-15)


def test_rope_invariants():
    d = 16
    x = RNG.standard_normal((5, 3, d))
    assert np.allclose(vlm.rope(x, np.zeros(5, int), 1e4), x, atol=1e-15)
    y = vlm.rope(x, np.arange(5) * 37, 1e4)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    q = RNG.standard_normal((1, 1, d))
    k = RNG.standard_normal((1, 1, d))
    dots = []
    for m, n in [(5, 2), (13, 10), (103, 100)]:
        dots.append(float((vlm.rope(q, np.array([m]), 1e4) * vlm.rope(k, np.array([n]), 1e4)).sum()))
    assert np.allclose(dots, dots[0], atol=1e-12)


# ----------------------------------------------------------------------------- vision encode
def test_patch_embed_equals_strided_conv():
    cfg = synth.VitConfig(hidden=16, heads=2, mlp=32, layers=0, patch=4, merge=2, out_hidden=8,
                          image_h=16, image_w=24)
    w = synth.vit_weights(cfg, seed=3)
    img = synth.image(1, 16, 24, seed=3)[0]
    ours = vlm.patch_embed(img, w, cfg)
    wconv = t64(w["patch.w"]).reshape(16, 4, 4, 3).permute(0, 3, 1, 2)
    conv = F.conv2d(t64(img).permute(2, 0, 1)[None], wconv, t64(w["patch.b"]), stride=4)
    ref = conv[0].permute(1, 2, 0).reshape(-1, 16).numpy() + w["pos"]
    assert np.allclose(ours, ref, atol=1e-12)


def test_merge_order_on_index_grid():
    cfg = synth.VitConfig(hidden=1, heads=1, mlp=1, layers=0, patch=1, merge=2, out_hidden=4,
                          image_h=4, image_w=6)
    # identity adapter: LN disabled by construction is impossible for width 1, so check the
    # concatenation order through the reshape the adapter applies
    idx = np.arange(24, dtype=float).reshape(24, 1)
    gh, gw, m = 4, 6, 2
    merged = idx.reshape(gh // m, m, gw // m, m, 1).transpose(0, 2, 1, 3, 4).reshape(6, 4)
    # token (i, j) = patches (2i,2j), (2i,2j+1), (2i+1,2j), (2i+1,2j+1) in row-major patch ids
    expect = np.array([[(2 * i) * gw + 2 * j, (2 * i) * gw + 2 * j + 1, (2 * i + 1) * gw + 2 * j,
                        (2 * i + 1) * gw + 2 * j + 1] for i in range(2) for j in range(3)], float)
    assert np.array_equal(merged, expect)
    # and through the oracle adapter: width-2 LN maps (a, b) to (+-1); Linear picks slots
    cfg2 = synth.VitConfig(hidden=2, heads=1, mlp=1, layers=0, patch=1, merge=2, out_hidden=8,
                           image_h=4, image_w=6)
    x = np.stack([np.arange(24.0), np.zeros(24)], 1)       # LN -> (+1, -1) for every patch
    x[::2, 1] = 1e3                                          # even patches flip to (-1, +1)
    w = {"merge.ln.g": np.ones(2), "merge.ln.b": np.zeros(2), "merge.w": np.eye(8), "merge.b": np.zeros(8)}
    out = vlm.merge_adapter(x, w, cfg2)
    first = out[:, 0::2]                                    # first LN component of each slot
    parity = np.where(expect % 2 == 0, -1.0, 1.0)
    assert np.allclose(first, parity, atol=1e-5)


def _torch_encoder_layer(w, cfg):
    layer = torch.nn.TransformerEncoderLayer(cfg.hidden, cfg.heads, cfg.mlp, dropout=0.0, activation="gelu",
                                             layer_norm_eps=cfg.eps, batch_first=True, norm_first=True,
                                             dtype=torch.float64)
    sd = {"self_attn.in_proj_weight": w["l0.qkv.w"], "self_attn.in_proj_bias": w["l0.qkv.b"],
          "self_attn.out_proj.weight": w["l0.o.w"], "self_attn.out_proj.bias": w["l0.o.b"],
          "linear1.weight": w["l0.fc1.w"], "linear1.bias": w["l0.fc1.b"],
          "linear2.weight": w["l0.fc2.w"], "linear2.bias": w["l0.fc2.b"],
          "norm1.weight": w["l0.ln1.g"], "norm1.bias": w["l0.ln1.b"],
          "norm2.weight": w["l0.ln2.g"], "norm2.bias": w["l0.ln2.b"]}
    layer.load_state_dict({k: t64(v) for k, v in sd.items()})
    return layer.eval()


def test_vit_layer_matches_torch_encoder_layer():
    cfg = synth.TINY_VIT
    w = synth.vit_weights(cfg, seed=0)
    x = RNG.standard_normal((cfg.n_patches, cfg.hidden))
    ours = vlm.vit_layer(x, w, 0, cfg)
    with torch.no_grad():
        ref = _torch_encoder_layer(w, cfg)(t64(x)[None])[0].numpy()
    assert vlm.max_rel_err(ours, ref) < 1e-12


def test_vit_layer_permutation_equivariant_and_rows():
    cfg = synth.TINY_VIT
    w = synth.vit_weights(cfg, seed=0)
    x = RNG.standard_normal((cfg.n_patches, cfg.hidden))
    perm = RNG.permutation(cfg.n_patches)
    a = vlm.vit_layer(x, w, 0, cfg)
    b = vlm.vit_layer(x[perm], w, 0, cfg)
    assert np.allclose(a[perm], b, atol=1e-12)
    rows = np.array([0, 5, 63])
    assert np.allclose(vlm.vit_layer(x, w, 0, cfg, rows=rows), a[rows], atol=1e-12)


def test_vit_encode_tokens_equals_full_encode():
    cfg = synth.VitConfig(hidden=64, heads=2, mlp=96, layers=2, patch=2, merge=2, out_hidden=64,
                          image_h=8, image_w=12)
    w = synth.vit_weights(cfg, seed=5)
    img = synth.image(1, 8, 12, seed=5)[0]
    full = vlm.vit_encode(img, w, cfg)
    toks = [0, 4, 5]
    assert np.allclose(vlm.vit_encode_tokens(img, w, cfg, toks), full[toks], atol=1e-12)


# ----------------------------------------------------------------------------- LLM
def _hf_llama(w, cfg):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(hidden_size=cfg.hidden, intermediate_size=cfg.inter, num_attention_heads=cfg.n_q,
                     num_key_value_heads=cfg.n_kv, head_dim=cfg.head_dim, num_hidden_layers=cfg.layers,
                     vocab_size=cfg.vocab, rms_norm_eps=cfg.eps, rope_theta=cfg.rope_theta,
                     tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).double().eval()
    sd = {"model.embed_tokens.weight": w["embed"], "model.norm.weight": w["norm.g"], "lm_head.weight": w["lm_head.w"]}
    for l in range(cfg.layers):
        p, q = f"l{l}.", f"model.layers.{l}."
        sd.update({q + "input_layernorm.weight": w[p + "rms1.g"], q + "post_attention_layernorm.weight": w[p + "rms2.g"],
                   q + "self_attn.q_proj.weight": w[p + "q.w"], q + "self_attn.k_proj.weight": w[p + "k.w"],
                   q + "self_attn.v_proj.weight": w[p + "v.w"], q + "self_attn.o_proj.weight": w[p + "o.w"],
                   q + "mlp.gate_proj.weight": w[p + "gate.w"], q + "mlp.up_proj.weight": w[p + "up.w"],
                   q + "mlp.down_proj.weight": w[p + "down.w"]})
    m.load_state_dict({k: t64(v) for k, v in sd.items()}, strict=False)
    return m


@pytest.mark.slow
def test_prefill_matches_hf_llama():
    cfg = synth.TINY_LLM
    w = synth.llm_weights(cfg, seed=0)
    vis = synth.vision_embeds(20, cfg.hidden, seed=4)
    ids = synth.text_ids(9, cfg.vocab, seed=2)
    logits, nxt, hid = vlm.llm_prefill(vis, ids, w, cfg, return_hidden=True)
    m = _hf_llama(w, cfg)
    emb = np.concatenate([vis, w["embed"][ids]], 0)
    with torch.no_grad():
        ref = m(inputs_embeds=t64(emb)[None]).logits[0].numpy()
    ours_all = vlm.lm_head(hid, w, cfg)
    # HF computes rotary angles in float32; that bounds the agreement near 1e-6
    assert vlm.max_rel_err(ours_all, ref) < 2e-5
    assert np.allclose(logits, ours_all[-1])
    assert nxt == int(np.argmax(ref[-1]))


def _decode_setup(cfg, n_vis=12, n_txt=5, steps=6, seed_blocks=5):
    w = synth.llm_weights(cfg, seed=0)
    vis = synth.vision_embeds(n_vis, cfg.hidden, seed=4)
    ids = synth.text_ids(n_txt, cfg.vocab, seed=2)
    return w, vis, ids


def _run_decode(w, vis, ids, cfg, steps, table, pool):
    s = len(vis) + len(ids)
    kv = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    _, tok = vlm.llm_prefill(vis, ids, w, cfg, kv=kv, table=table)
    toks, logs = [tok], []
    for t in range(steps):
        lg, nx = vlm.llm_decode_step(np.array([toks[-1]]), np.array([s + t]), table[None], kv, w, cfg)
        logs.append(lg[0])
        toks.append(int(nx[0]))
    return toks, logs


def test_decode_step_equals_prefill_recompute():
    cfg = synth.TINY_LLM
    w, vis, ids = _decode_setup(cfg)
    steps = 6
    s = len(vis) + len(ids)
    table, pool = synth.block_tables([s + steps], cfg.block, seed=5)
    toks, logs = _run_decode(w, vis, ids, cfg, steps, table[0], pool)
    for t in range(steps):
        ext = np.concatenate([ids, np.array(toks[:t + 1], np.int32)])
        ref, _ = vlm.llm_prefill(vis, ext, w, cfg)
        assert vlm.max_rel_err(logs[t], ref) < 1e-10


def test_paged_cache_invariant_to_block_permutation():
    cfg = synth.TINY_LLM
    w, vis, ids = _decode_setup(cfg)
    s = len(vis) + len(ids)
    t1, pool = synth.block_tables([s + 4], cfg.block, seed=5, num_blocks=9)
    t2, _ = synth.block_tables([s + 4], cfg.block, seed=6, num_blocks=9)
    assert not np.array_equal(t1, t2)
    a = _run_decode(w, vis, ids, cfg, 4, t1[0], pool)
    b = _run_decode(w, vis, ids, cfg, 4, t2[0], pool)
    assert a[0] == b[0] and all(np.array_equal(x, y) for x, y in zip(a[1], b[1]))


def test_batched_decode_equals_single_sequences():
    cfg = synth.TINY_LLM
    w = synth.llm_weights(cfg, seed=0)
    lens = [7, 19, 16]
    tables, pool = synth.block_tables([n + 1 for n in lens], cfg.block, seed=8)
    kv = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    firsts = []
    for b, n in enumerate(lens):
        vis = synth.vision_embeds(n - 3, cfg.hidden, seed=10 + b)
        ids = synth.text_ids(3, cfg.vocab, seed=20 + b)
        firsts.append(vlm.llm_prefill(vis, ids, w, cfg, kv=kv, table=tables[b])[1])
    kv_copy = vlm.PagedKV(cfg.layers, pool, cfg.n_kv, cfg.block, cfg.head_dim)
    kv_copy.k[:], kv_copy.v[:] = kv.k, kv.v
    lg, nx = vlm.llm_decode_step(np.array(firsts), np.array(lens), tables, kv, w, cfg)
    for b in range(3):
        lg1, nx1 = vlm.llm_decode_step(np.array(firsts[b:b + 1]), np.array(lens[b:b + 1]), tables[b:b + 1], kv_copy, w, cfg)
        assert np.allclose(lg[b], lg1[0], atol=1e-13) and nx[b] == nx1[0]


def test_layer_rows_equal_full_prefill_layer():
    cfg = synth.LlmConfig(hidden=64, n_q=4, n_kv=2, head_dim=16, inter=96, vocab=50, layers=1)
    w = synth.llm_weights(cfg, seed=1)
    vis = synth.vision_embeds(15, 64, seed=1)
    ids = synth.text_ids(4, 50, seed=1)
    _, _, hid = vlm.llm_prefill(vis, ids, w, cfg, return_hidden=True)
    x = np.concatenate([vis, w["embed"][ids]], 0)
    rows = np.array([0, 7, 18])
    out, k, v = vlm.llm_layer_rows(x, w, 0, cfg, rows)
    assert np.allclose(out, hid[rows], atol=1e-13)


def test_greedy_ties_lowest_index():
    assert vlm.greedy(np.array([0.1, 0.7, 0.7, -1.0])) == 1
    assert list(vlm.greedy(np.array([[3.0, 3.0], [0.0, 1.0]]))) == [0, 1]


# ----------------------------------------------------------------------------- scheduling formulas
def test_eq5_printed_values():
    g = GOLDEN["eq5_sm_assignment"]
    for c in g["cases"]:
        got = [sched.decode_share(c["sm_op"], c["alpha"], g["sm_min"], n) for n in c["n_pend"]]
        assert got == c["sm_dec"]


def test_eq7_worked_example():
    g = GOLDEN["eq7_worked_example"]
    k = g["k"]
    layers = 64
    cur0 = g["forwarding_model_layer_1idx"] - 1        # 0-indexed layer being forwarded
    assert cur0 % k + 1 == g["forwarding_physical_slot_1idx"]
    # the two layers that finished before it free their slots and pull (cur + K) mod L
    for (model1, slot1), finished0 in zip(g["swapping_in_1idx"], [cur0 - 2, cur0 - 1]):
        nxt = sched.next_layer(finished0, k, layers)
        assert nxt + 1 == model1 and finished0 % k + 1 == slot1
    assert sched.next_layer(63, 2, 64) == 1               # wraps into the next pass


def test_ring_slots_worked_by_hand():
    # L = 5, K = 3, one pass: slot 0 holds 0 then 3, and after 3 takes 1; slot 1 holds 1, 4, then 2;
    # slot 2 holds 2, then 0
    assert sched.ring_slots(5, 3, 1) == [1, 2, 0]
    assert sched.ring_slots(5, 3, 2) == [2, 0, 1]
    # K divides L: every slot keeps its residue class, so the map never moves
    assert sched.ring_slots(6, 3, 4) == [0, 1, 2]
    assert sched.ring_slots(64, 2, 3) == [0, 1]
    # after any number of passes the slots hold the next pass's first K layers
    for n_layers, k in [(5, 2), (5, 3), (7, 4), (32, 3)]:
        for passes in range(4):
            assert sorted(sched.ring_slots(n_layers, k, passes)) == list(range(k))


def test_eq8_printed_bound_and_closed_form():
    g = GOLDEN["eq8_bandwidth"]
    need = [sched.offload_min_bandwidth(g["size_gb"], t, g["vit_layers"], 2) for t in g["t_fwd_s"]]
    assert max(need) == pytest.approx(g["max_needed_gbps"])
    assert max(need) < g["pcie4_gbps"]
    r = np.random.default_rng(7)
    for _ in range(200):
        L = int(r.integers(4, 80))
        K = int(r.integers(2, L - 1))
        S, T = float(r.uniform(1, 10)), float(r.uniform(0.1, 2))
        bmin = sched.offload_min_bandwidth(S, T, L, K)
        assert sched.offload_ok(S, T, bmin * (1 + 1e-9), L, K)
        assert not sched.offload_ok(S, T, bmin * (1 - 1e-6), L, K)


def test_eq6_against_printed_mg1_table():
    g = GOLDEN["table_mg1"]
    for lam, t, util, pred in zip(g["lambda"], g["mean_t_s"], g["utilization"], g["mg1_prediction_s"]):
        assert abs(lam * t - util) <= 0.0051 + 1e-9 or (lam, util) == (0.6, 0.86)
        if pred is None:
            continue
        det = sched.mg1_wait(lam, t, t * t)          # E[T^2] >= E[T]^2: deterministic service is the floor
        assert det <= pred <= det * 1.08


def test_eq1_to_eq4_partition_search():
    shares = [32, 64, 96, 128, 160, 192, 224]
    # vision/prefill speed up with more units; decode time depends only on its own share
    t_v = {p: 2.0 * 256 / p for p in shares}
    t_p = {p: 1.0 * 256 / p for p in shares}
    t_d = {p: 0.01 * 256 / (256 - p) for p in shares}
    pv, pp, lat = sched.optimal_partition(shares, t_v, t_p, t_d, t_d, 40)
    grid = {(a, b): t_v[a] + t_p[b] + (t_v[a] * t_d[a] + t_p[b] * t_d[b]) / (t_v[a] + t_p[b]) * 40
            for a in shares for b in shares}
    best = min(grid, key=grid.get)
    assert (pv, pp) == best and lat == pytest.approx(grid[best])
    assert sched.e2e_latency(3.0, 1.0, 0.02, 0.02, 50) == pytest.approx(3.0 + 1.0 + 0.02 * 50)
    assert sched.throughput(0.8, 0.3) == pytest.approx(1 / 1.1)
    pts = [(1.0, 1.0, "a"), (2.0, 2.0, "b"), (1.5, 0.5, "c"), (3.0, 2.0, "d")]
    assert [p[2] for p in sched.pareto_front(pts)] == ["a", "b"]


def test_table4_and_offload_table_arithmetic():
    g = GOLDEN["table_linear_corun"]
    assert g["decode"]["solo_ms"] + g["vision"]["solo_ms"] == pytest.approx(1288.1)
    assert g["decode"]["dram_gbps"] / g["a6000_peak_gbps"] == pytest.approx(0.83, abs=0.005)
    o = GOLDEN["table_offload"]
    steps = np.diff(o["mem_mb"])
    assert np.allclose(steps, steps[0], atol=0.2)          # one physical layer per extra K
    assert 1 - o["mem_mb"][0] / o["raw_mem_mb"] > 0.9


def test_max_rel_err_flags_known_perturbations():
    """The parity metric itself: max|g - o| / max|o| over one tensor, checked on values whose
    answer is known by hand, and shown to flag each kind of mistake a parity test must catch."""
    ref = np.arange(-12.0, 12.0).reshape(4, 6)                 # max |ref| = 12
    assert vlm.max_rel_err(ref, ref) == 0.0
    got = ref.copy()
    got[1, 3] += 0.3                                            # one element off by 0.3
    assert vlm.max_rel_err(got, ref) == pytest.approx(0.3 / 12.0, rel=1e-12)
    assert vlm.max_rel_err(3.5 * got, 3.5 * ref) == pytest.approx(0.3 / 12.0, rel=1e-12)   # scale-free
    assert vlm.max_rel_err(np.zeros(3), np.zeros(3)) == 0.0    # an all-zero reference is absolute
    assert vlm.max_rel_err(np.full(3, 0.5), np.zeros(3)) == 0.5
    # the 2e-2 bound: a 2.5% error in the largest element fails it, a 1% one passes
    big = ref.copy()
    big[0, 0] *= 1.025
    small = ref.copy()
    small[0, 0] *= 1.01
    assert vlm.max_rel_err(big, ref) > 2e-2 > vlm.max_rel_err(small, ref)
    # a flipped sign, a transposed operand, a dropped term and a shifted index are all far above it
    rng = np.random.default_rng(0)
    a = rng.standard_normal((8, 8))
    b = rng.standard_normal((8, 8))
    flipped = a.copy()
    flipped[2, 5] = -flipped[2, 5]
    assert vlm.max_rel_err(flipped, a) > 2e-2 or a[2, 5] == 0
    assert vlm.max_rel_err(a.T @ b, a @ b) > 2e-2
    assert vlm.max_rel_err(a @ b, a @ b + 0.1 * b) > 2e-2
    assert vlm.max_rel_err(np.roll(a, 1, axis=0), a) > 2e-2
    # NaN anywhere in the output is never within tolerance
    nan = a.copy()
    nan[3, 3] = np.nan
    assert not vlm.max_rel_err(nan, a) < 2e-2


def test_bf16_store_rounding():
    """bf16_store against torch's float32 -> bfloat16 conversion (an independent implementation of
    round-to-nearest-even) and against hand-worked ties."""
    import torch
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        [0.0, -0.0, 1e-40, -3e-39, np.inf, -np.inf, 3.3895e38, 1.0, -2.5]]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy().astype(np.float64)
    got = vlm.bf16_store(x)
    assert np.array_equal(got, want)
    one = 1.0
    assert vlm.bf16_store(one + 2.0 ** -8) == 1.0                   # halfway, to the even neighbour 1
    assert vlm.bf16_store(one + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6    # halfway, to the even neighbour above
    assert vlm.bf16_store(one + 2.0 ** -8 + 2.0 ** -20) == 1.0 + 2.0 ** -7   # just past halfway: up
    assert np.isnan(vlm.bf16_store(np.nan))
    assert np.array_equal(vlm.bf16_store(got), got)                  # idempotent


def test_bf16_store_points_in_the_llm():
    """The stored tensors of the bf16-storage reading: per layer the normed input, the q / k / v
    projections, the rotated q and k, the attention output, the MLP's normed input and hidden
    activation; then the final normed row (prefill: last row only)."""
    cfg = synth.TINY_LLM
    w = synth.llm_weights(cfg, seed=0)
    seen = []

    def store(t):
        seen.append(np.shape(t))
        return t
    vis = synth.vision_embeds(8, cfg.hidden)
    ids = synth.text_ids(5, cfg.vocab)
    s, H, d = 13, cfg.hidden, cfg.head_dim
    exact = vlm.llm_prefill(vis, ids, w, cfg)[0]
    got = vlm.llm_prefill(vis, ids, w, cfg, store=store)[0]
    assert np.array_equal(got, exact)                                # recording changes nothing
    per_layer = [(s, H), (s, cfg.n_q * d), (s, cfg.n_q, d), (s, cfg.n_kv * d), (s, cfg.n_kv, d), (s, cfg.n_kv * d),
                 (s, cfg.n_q, d), (s, H), (s, cfg.inter)]
    assert seen == per_layer * cfg.layers + [(1, H)]
    # bf16 storage moves the logits by a bf16-sized amount, no more
    rounded = vlm.llm_prefill(vis, ids, w, cfg, store=vlm.bf16_store)[0]
    assert 1e-4 < vlm.max_rel_err(rounded, exact) < 2e-2
