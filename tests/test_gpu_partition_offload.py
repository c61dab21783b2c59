"""CU partitions (Sec. 3.2.2) and vision-encoder layer offload (Sec. 3.5, Eq. 7) on the GPU.

* A stage's partition stream runs only on the CUs of its mask: balanced over the 8 XCDs and
  their shader engines, disjoint from the complementary mask, and full masks see all 256 CUs.
* Work switched between partition streams keeps its order (decode steps that read the KV
  written by the previous step on another partition give bit-identical logits).
* Invalid masks are rejected; the whole-GPU mask has a stream per stage.
* Encoding with K = 2 or 3 device slots streamed from pinned memory (including a deliberately
  delayed preload) is bit-identical to the resident model, across consecutive calls whose ring
  wraps into the next pass; the encoder with 2x2 merge matches the oracle.
"""
import numpy as np
import pytest

from oracle import sched as osched
from oracle import vlm
from paper_2509_21301_amd import synth
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu

VIT5 = synth.VitConfig(hidden=256, heads=4, mlp=1024, layers=5, patch=4, merge=2, out_hidden=256,
                       image_h=32, image_w=48, name="vit5_merge")


def test_whole_gpu_mask_has_a_stream_per_stage(gpu_lib):
    # two stages may both hold the whole GPU for a pass; sharing one stream would queue one
    # stage's pass behind the other's
    nova = gpu_lib
    full = [0xFFFFFFFF] * 8
    streams = {nova.set_stage_partition(st, full).cuda_stream
               for st in (nova.STAGE_ENCODE, nova.STAGE_PREFILL, nova.STAGE_DECODE)}
    assert len(streams) == 3
    a = nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(96, 0)).cuda_stream
    b = nova.set_stage_partition(nova.STAGE_ENCODE, nova.make_cu_mask(96, 0)).cuda_stream
    assert a == b                      # a partial mask is one stream, whoever holds it
    assert nova.set_stage_partition(nova.STAGE_DECODE, full).cuda_stream in streams


def test_partition_streams_stay_on_their_cus(gpu_lib):
    nova = gpu_lib
    full = nova.cu_probe(nova.set_stage_partition(nova.STAGE_ENCODE, [0xFFFFFFFF] * 8))
    assert len(full) == nova.device_cus() == 256
    for n_cus, first in [(64, 0), (192, 8), (32, 28)]:
        units = nova.cu_probe(nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(n_cus, first)))
        assert len(units) == n_cus
        per_xcd = {}
        per_se = {}
        for x, se, cu in units:
            per_xcd[x] = per_xcd.get(x, 0) + 1
            per_se[(x, se)] = per_se.get((x, se), 0) + 1
        assert sorted(per_xcd) == list(range(8)) and set(per_xcd.values()) == {n_cus // 8}
        if n_cus // 8 % 4 == 0:
            assert set(per_se.values()) == {n_cus // 32}
    a = nova.cu_probe(nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(64, 0)))
    b = nova.cu_probe(nova.set_stage_partition(nova.STAGE_ENCODE, nova.make_cu_mask(192, 8)))
    assert not (a & b) and len(a | b) == 256


def test_invalid_masks_rejected(gpu_lib):
    nova = gpu_lib
    with pytest.raises(nova.NovaError):
        nova.set_stage_partition(nova.STAGE_DECODE, [0] * 8)
    with pytest.raises(nova.NovaError):            # XCD 0 would have no CU (bit i -> XCD i % 8)
        nova.set_stage_partition(nova.STAGE_DECODE, [0xFEFEFEFE] * 8)
    with pytest.raises(nova.NovaError):
        nova.set_stage_partition(7, [0xFFFFFFFF] * 8)
    with pytest.raises(nova.NovaError):
        nova.make_cu_mask(12, 0)


def test_stage_switch_keeps_order(gpu_lib):
    import torch
    nova = gpu_lib
    ref = sc.oracle_tiny(decode_steps=6)
    cfg = synth.TINY_LLM
    llm = nova.Llm(cfg, ref["wl"], act=nova.ACT_BF16)

    def run(switch):
        kv = nova.KvPool(llm, ref["pool"])
        table = torch.from_numpy(ref["table"]).cuda()
        vis = torch.from_numpy(ref["vis"]).cuda().to(torch.bfloat16)
        ids = torch.from_numpy(ref["ids"]).cuda()
        s0 = nova.set_stage_partition(nova.STAGE_PREFILL, [0xFFFFFFFF] * 8)
        tok = llm.prefill(vis, ids, table[0], kv, stream=s0)
        s0.synchronize()
        logs = []
        for t in range(6):
            mask = nova.make_cu_mask(64 if t % 2 else 192, 0 if t % 2 else 8) if switch else [0xFFFFFFFF] * 8
            st = nova.set_stage_partition(nova.STAGE_DECODE, mask)
            lg = torch.empty(1, cfg.vocab, dtype=torch.float32, device="cuda")
            pos = torch.tensor([ref["s"] + t], dtype=torch.int32, device="cuda")
            tok = llm.decode(tok, pos, table, kv, max_ctx=ref["s"] + 6, logits=lg, stream=st)
            logs.append(lg)
        torch.cuda.synchronize()
        return [l.cpu().numpy() for l in logs]

    a, b = run(False), run(True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.fixture(scope="module")
def vit5():
    w = synth.vit_weights(VIT5, seed=3)
    imgs = synth.image(2, VIT5.image_h, VIT5.image_w, seed=7)
    ref = np.stack([vlm.vit_encode(imgs[i], w, VIT5) for i in range(2)])
    return w, imgs, ref


@pytest.mark.parametrize("act", ["bf16", "f32"])
def test_merge_encoder_matches_oracle(gpu_lib, vit5, act):
    import torch
    nova = gpu_lib
    w, imgs, ref = vit5
    a = nova.ACT_F32 if act == "f32" else nova.ACT_BF16
    vit = nova.Vit(VIT5, w, act=a)
    out = vit.encode(torch.from_numpy(imgs).cuda().to(torch.bfloat16)).float().cpu().numpy()
    tol = sc.TOL_F32 if act == "f32" else sc.TOL_BF16
    for i in range(2):
        assert vlm.max_rel_err(out[i], ref[i]) < tol


@pytest.mark.parametrize("k_slots", [2, 3])
def test_offload_bit_identical_to_resident(gpu_lib, vit5, k_slots):
    import torch
    nova = gpu_lib
    w, imgs, _ = vit5
    px = torch.from_numpy(imgs).cuda().to(torch.bfloat16)
    resident = nova.Vit(VIT5, w).encode(px).cpu()
    off = nova.Vit(VIT5, w, n_slots=k_slots)
    # preload the first K layers on a stream that is kept busy first, so that the copies land
    # late and the encoder must wait on the slot events
    slow = torch.cuda.Stream()
    with torch.cuda.stream(slow):
        big = torch.randn(4096, 4096, device="cuda")
        for _ in range(8):
            big = big @ big * 1e-3
    for layer in range(k_slots):
        off.prefetch(layer, stream=slow)
    for call in range(3):            # the ring wraps: each call's tail loads the next call's head
        got = off.encode(px).cpu()
        assert torch.equal(got, resident), f"call {call}"
        # one copy per layer per call after the K preloads, slots rotating as Eq. 7 says (K = 3
        # does not divide L = 5)
        slots, copies = off.offload_state()
        assert copies == k_slots + (call + 1) * VIT5.layers
        assert slots == osched.ring_slots(VIT5.layers, k_slots, call + 1)
    torch.cuda.synchronize()


def test_complementary_partitions_run_concurrently(gpu_lib):
    """Encode on 192 CUs and decode on the complementary 64, launched together, overlap: the
    span from the first start to the last end is well below the two solo times added (the
    hardware queues of complementary masks sit on different dispatch pipes)."""
    import dataclasses

    import torch

    import bench
    nova = gpu_lib
    vc = dataclasses.replace(synth.VIT_1008, layers=4)
    lc = dataclasses.replace(synth.LLM_28, layers=2)
    vit = bench.build_vit(nova, vc, "cuda")
    llm = bench.build_llm(nova, lc, "cuda")
    px = torch.from_numpy(synth.image(4, vc.image_h, vc.image_w, seed=1)).to("cuda", torch.bfloat16).contiguous()
    enc_out = torch.empty(vit.out_shape(4), dtype=torch.bfloat16, device="cuda")
    ctx = 1500
    tables, pool = synth.block_tables([ctx + 1] * 8, lc.block, seed=5)
    kv = nova.KvPool(llm, pool)
    tab = torch.from_numpy(tables).cuda()
    ids = torch.from_numpy(synth.text_ids(8, lc.vocab, seed=9)).cuda()
    pos = torch.full((8,), ctx, dtype=torch.int32, device="cuda")
    s_e = nova.set_stage_partition(nova.STAGE_ENCODE, nova.make_cu_mask(192, 8))
    s_d = nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(64, 0))

    def encode():
        vit.encode(px, out=enc_out, stream=s_e)

    def decode(n):
        for _ in range(n):
            llm.decode(ids, pos, tab, kv, ctx + 1, stream=s_d)

    def timed(fn, stream):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b)

    t_e = timed(encode, s_e)
    t_step = timed(lambda: decode(4), s_d) / 4
    n = max(4, int(round(t_e / t_step)))
    t_d = timed(lambda: decode(n), s_d)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    ev[0].record(s_e)
    ev[1].record(s_d)
    encode()
    decode(n)
    ev[2].record(s_e)
    ev[3].record(s_d)
    torch.cuda.synchronize()
    start = min(ev[0], ev[1], key=lambda e: ev[0].elapsed_time(e))
    span = max(start.elapsed_time(ev[2]), start.elapsed_time(ev[3]))
    print(f"[corun] encode {t_e:.2f} ms, decode x{n} {t_d:.2f} ms, together {span:.2f} ms")
    assert span < 0.8 * (t_e + t_d)
