"""Benchmark of the single-GPU VLM serving hot path on MI355X.

Headline: vision-encode throughput (patches/s) of the 32-layer, 1280-wide ViT on 1008x1008
images (5184 patches each, 2x2 merge to 3584) at batch 8 on all 256 CUs.  The same JSON line
carries per-stage throughput (encode patches/s at batch 1/4/8, prefill tok/s of a 1500-token
prompt, decode tok/s at batch 1/8/32 on the 28-layer GQA decoder), each stage's throughput
against its CU share (XCD-balanced masks of 32..256 CUs), decode co-running with encode and
with prefill on complementary partitions, the roofline position of the dominant kernel family,
and the oracle's CPU time on a bounded sample.

All inputs are seeded synthetic data of the workload shapes; weights are random N(0, 0.02)
bf16 generated on the device.  Usage: python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------- model builders
def random_blob(nbytes, offsets, norm_idx, device, gen, std=0.02):
    """A packed weight blob of N(0, std) bf16 with the norm-gain tensors set to 1 + N(0, 0.2)."""
    import torch
    t = (torch.randn(nbytes // 2, generator=gen, device=device, dtype=torch.float32) * std).to(torch.bfloat16)
    return t


def build_vit(nova, cfg, device, seed=0, n_slots=0):
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    (eo, eb), (lo, lb), (ho, hb) = nova.vit_layouts(cfg)
    H = cfg.hidden
    emb = random_blob(eb, eo, [], device, gen)
    layers = random_blob(lb * cfg.layers, lo, [], device, gen)
    head = random_blob(hb, ho, [], device, gen)
    lv = layers.view(cfg.layers, lb // 2)
    for i in (0, 6):      # ln1.g, ln2.g
        lv[:, lo[i] // 2: lo[i] // 2 + H] = 1.0
    head[ho[0] // 2: ho[0] // 2 + H] = 1.0
    if n_slots > 0:
        host = torch.empty(layers.numel(), dtype=torch.bfloat16, pin_memory=True)
        host.copy_(layers)
        layers = host
    return nova.Vit(cfg, None, blobs=(emb, layers, head, lb), n_slots=n_slots)


def build_llm(nova, cfg, device, seed=1):
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    (lo, lb), (ho, hb) = nova.llm_layouts(cfg)
    H = cfg.hidden
    layers = random_blob(lb * cfg.layers, lo, [], device, gen)
    lv = layers.view(cfg.layers, lb // 2)
    for i in (0, 3):      # rms1.g, rms2.g
        lv[:, lo[i] // 2: lo[i] // 2 + H] = 1.0
    head = random_blob(hb, ho, [], device, gen)
    head[ho[0] // 2: ho[0] // 2 + H] = 1.0
    embed = (torch.randn(cfg.vocab * H, generator=gen, device=device) * 0.02).to(torch.bfloat16).view(cfg.vocab, H)
    return nova.Llm(cfg, None, blobs=(embed, layers, head, lb))


# ----------------------------------------------------------------------------- work counts
def vit_flops(cfg, batch):
    """Algorithmic FLOPs of one encode pass: GEMMs (patch embed, 4 linears per layer, adapter) and attention."""
    n, H, I = cfg.n_patches, cfg.hidden, cfg.mlp
    lin_layer = 2 * n * H * (3 * H + H + I + I)
    attn_layer = 4 * n * n * H
    embed = 2 * n * cfg.patch_dim * H
    merge = 2 * cfg.n_out * (cfg.merge ** 2 * H) * cfg.out_hidden
    gemm = cfg.layers * lin_layer + embed + merge
    return batch * gemm, batch * cfg.layers * attn_layer


def prefill_flops(cfg, s):
    H, d = cfg.hidden, cfg.head_dim
    lin = 2 * s * H * ((cfg.n_q + 2 * cfg.n_kv) * d + cfg.n_q * d + 3 * cfg.inter) * cfg.layers
    attn = 2 * s * s * cfg.n_q * d * cfg.layers          # causal: half of 4 S^2 n_q d
    head = 2 * H * cfg.vocab
    return lin + head, attn


def decode_bytes(cfg, batch, ctx):
    """Algorithmic HBM bytes of one decode step: every weight once plus each sequence's K/V."""
    H, d, I = cfg.hidden, cfg.head_dim, cfg.inter
    w_layer = (H * (cfg.n_q + 2 * cfg.n_kv) * d + H * cfg.n_q * d + 3 * H * I + 2 * H) * 2
    weights = cfg.layers * w_layer + (cfg.vocab * H + H) * 2 + batch * H * 2
    kv = batch * ctx * cfg.layers * cfg.n_kv * d * 2 * 2
    return weights, kv


# ----------------------------------------------------------------------------- HBM traffic
def gemm_traffic():
    """HBM bytes per GEMM call of the encode pass (one call of the GEMM routine, the unit timed
    below; the split problems launch two kernels per call), from the committed rocprofv3 PMC summary
    (FETCH_SIZE and WRITE_SIZE, each scaled by its reading for a plain 1 GiB copy); None when the
    summary is missing or the GEMM source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "encode_gemm_hbm_traffic.md")
    src = os.path.join(ROOT, "paper_2509_21301_amd", "csrc", "k_gemm.hip")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.strip().startswith("- `"):
            k, v = line.strip()[3:].split("`", 1)
            vals[k] = v.strip(" :`")
    want = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if vals.get("kernel_source_sha256") != want or "traffic_bytes_per_launch" not in vals:
        return None
    return int(float(vals["traffic_bytes_per_launch"]))


# ----------------------------------------------------------------------------- timing helpers
def time_passes(torch, fn, reps, stream):
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def time_each(torch, fn, reps, stream):
    """Per-pass times (ms), each pass between its own pair of HIP events on the stream."""
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record(stream)
    for i in range(reps):
        fn()
        ev[i + 1].record(stream)
    ev[-1].synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]


def spread(ts):
    """Median, 10th and 90th percentile of pass times (ms)."""
    q = np.percentile(np.asarray(ts), [50, 10, 90])
    return {"ms": round(float(q[0]), 3), "ms_p10": round(float(q[1]), 3), "ms_p90": round(float(q[2]), 3)}


class Stages:
    """The three stage workloads on one GPU, each callable on a given stream."""

    def __init__(self, nova, torch, synth, device, enc_batch):
        self.nova, self.torch = nova, torch
        self.vc, self.lc = synth.VIT_1008, synth.LLM_28
        log("building ViT-32 (1008x1008) and LLM-28 random weights on the device")
        self.vit = build_vit(nova, self.vc, device)
        self.llm = build_llm(nova, self.lc, device)
        img = synth.image(enc_batch, self.vc.image_h, self.vc.image_w, seed=1)
        self.pixels = torch.from_numpy(img).to(device, torch.bfloat16).contiguous()
        self.enc_out = torch.empty(self.vit.out_shape(enc_batch), dtype=torch.bfloat16, device=device)
        # prefill: 1300 vision embeddings + 200 text ids
        nv, nt = synth.LLM_VISION_TOKENS, synth.LLM_TEXT_TOKENS
        self.s = nv + nt
        self.vis = torch.from_numpy(synth.vision_embeds(nv, self.lc.hidden)).to(device, torch.bfloat16)
        self.ids = torch.from_numpy(synth.text_ids(nt, self.lc.vocab)).to(device)
        # KV pool for 32 sequences of up to 1500 + 64 tokens, plus one prefill sequence
        self.ctx_max = self.s + synth.LLM_DECODE_STEPS
        self.bmax = 32
        tables, pool = synth.block_tables([self.ctx_max] * (self.bmax + 1), self.lc.block, seed=5)
        self.pool = pool
        self.kv = nova.KvPool(self.llm, pool)
        g = torch.Generator(device=device)
        g.manual_seed(7)
        self.kv.k.copy_((torch.randn(self.kv.k.numel(), generator=g, device=device) * 0.5).to(self.kv.k.dtype))
        self.kv.v.copy_((torch.randn(self.kv.v.numel(), generator=g, device=device) * 0.5).to(self.kv.v.dtype))
        self.tables = torch.from_numpy(tables).to(device)
        self.pre_table = self.tables[self.bmax]
        self.dec_ids = torch.from_numpy(synth.text_ids(self.bmax, self.lc.vocab, seed=9)).to(device)
        self.dec_pos = torch.full((self.bmax,), self.s, dtype=torch.int32, device=device)
        self.next_ids = torch.empty(self.bmax, dtype=torch.int32, device=device)
        self.pre_next = torch.empty(1, dtype=torch.int32, device=device)
        # warm every workspace once
        torch.cuda.synchronize()

    def encode(self, batch=None, stream=None):
        px = self.pixels if batch is None else self.pixels[:batch]
        out = self.enc_out if batch is None else self.enc_out[:batch]
        self.vit.encode(px, out=out, stream=stream)

    def prefill(self, stream=None):
        self.llm.prefill(self.vis, self.ids, self.pre_table, self.kv, next_id=self.pre_next, stream=stream)

    def decode(self, batch, stream=None):
        self.llm.decode(self.dec_ids[:batch], self.dec_pos[:batch], self.tables[:batch], self.kv, self.ctx_max,
                        next_ids=self.next_ids[:batch], stream=stream)


class ServingSetup:
    """The screenshot workload: a 1092x2408 image (13416 patches, 3354 merged tokens) through the
    same 32-layer encoder (its own position table), prompts of 3354 + 150..300 tokens.  With
    n_slots > 0 the encoder's layers stay in pinned host memory and stream through that many
    device slots (Sec. 3.5); kv_blocks sizes the paged KV pool."""

    def __init__(self, nova, torch, synth, st, n_slots=0, kv_blocks=30000):
        self.nova, self.torch, self.synth, self.st = nova, torch, synth, st
        cfg = synth.VIT_SCREEN
        gen = torch.Generator(device="cuda")
        gen.manual_seed(11)
        (eo, eb), _, _ = nova.vit_layouts(cfg)
        emb = random_blob(eb, eo, [], "cuda", gen)
        layers = st.vit.layers
        if n_slots > 0:
            layers = torch.empty(st.vit.layers.numel(), dtype=torch.bfloat16, pin_memory=True)
            layers.copy_(st.vit.layers)
        self.n_slots, self.kv_blocks = n_slots, kv_blocks
        self.vit = nova.Vit(cfg, None, blobs=(emb, layers, st.vit.head, st.vit.layer_bytes), n_slots=n_slots)
        img = synth.image(1, cfg.image_h, cfg.image_w, seed=21)
        self.pixels = torch.from_numpy(img).to("cuda", torch.bfloat16).contiguous()
        self.vis = torch.empty(self.vit.out_shape(1), dtype=torch.bfloat16, device="cuda")
        nt = 225
        self.ids = torch.from_numpy(synth.text_ids(nt, st.lc.vocab, seed=22)).cuda()
        s = cfg.n_out + nt
        self.max_blocks = (cfg.n_out + 300 + 48 + 15) // 16
        tables, pool = synth.block_tables([s], 16, seed=23, num_blocks=kv_blocks)
        self.kv = nova.KvPool(st.llm, pool)
        self.table = torch.from_numpy(tables[0]).cuda()

    def encode(self, stream):
        self.vit.encode(self.pixels, out=self.vis, stream=stream)

    def prefill(self, stream):
        self.st.llm.prefill(self.vis[0], self.ids, self.table, self.kv, stream=stream)

    def serve(self, kw, trace, keep_log=False):
        from paper_2509_21301_amd import serve
        srv = serve.Server(self.vit, self.st.llm, self.kv, self.pixels, max_blocks=self.max_blocks, **kw)
        res = srv.run(trace)
        if keep_log and srv.partition_log:
            t0 = min(r.t_arrive for r in trace)
            res["partition_timeline"] = [[round((t - t0) * 1e3, 2), st, cus] for t, st, cus in srv.partition_log]
            res["arrivals_ms"] = [round(r.arrival * 1e3, 1) for r in trace]
        return res


# ----------------------------------------------------------------------------- serving runs
def serving_modes(sched, curves, out_len, rate, adaptive, adaptive32=None):
    """The systems compared on one trace: Nova at the rate's Pareto point (Eq. 1 + Eq. 6) and with
    the Eq. 5 adaptation (parameters from adaptive_params), time slicing decode-first and
    prefill-first, the PF-Limit baseline (prefill-first, decode once more than 5 wait; Sec. 5.1),
    and unpartitioned streams (Multi-Stream)."""
    rv, rp, _ = sched.best_under_load(sched.on_granule(curves), out_len, rate)
    a = adaptive
    modes = [("nova_rate_static", dict(mode="nova", decode_cus=(rv, rp))),
             ("nova_adaptive", dict(mode="nova", decode_cus=(a["sm_op_v"], a["sm_op_p"]),
                                    alpha=(a["alpha_v"], a["alpha_p"]), minimum=a["sm_min"]))]
    if adaptive32 is not None:
        # the same adaptation on shares of whole mask words (32 CUs): at most 7 partition pairs,
        # so the stream pool never has to create streams while serving
        b = adaptive32
        modes.append(("nova_adaptive_g32", dict(mode="nova", decode_cus=(b["sm_op_v"], b["sm_op_p"]),
                                                alpha=(b["alpha_v"], b["alpha_p"]), minimum=b["sm_min"], granule=32)))
    return modes + [
        ("time_sliced_decode_first", dict(mode="time_sliced", slice_order="decode_first")),
        ("time_sliced_prefill_first", dict(mode="time_sliced", slice_order="prefill_first")),
        ("pf_limit", dict(mode="time_sliced", slice_order="prefill_first", decode_limit=5)),
        ("multi_stream", dict(mode="multi_stream"))]


def run_serving(serve, sched, srv, curves, out_len, rates, seeds, window, modes=None, timeline_at=None):
    """Every mode on the same Poisson traces (rate x seed); per (mode, rate) the mean and spread
    over seeds, the better of the two time-sliced orders, and Eq. 6 beside the measured wait."""
    grid = sorted(set([0.25, 0.5, 1, 1.5, 2, 3, 4, 5, 6, 7, 8] + list(rates)))
    adaptive = sched.adaptive_params(curves, out_len, grid)
    adaptive32 = sched.adaptive_params(curves, out_len, grid, granule=32) if modes and "nova_adaptive_g32" in modes else None
    log(f"adaptive Eq. 5 parameters: SM_op {adaptive['sm_op_v']}/{adaptive['sm_op_p']}, alpha "
        f"{adaptive['alpha_v']}/{adaptive['alpha_p']}, SM_min {adaptive['sm_min']}")
    runs = []
    for rate in rates:
        for seed in seeds:
            for mode, kw in serving_modes(sched, curves, out_len, rate, adaptive, adaptive32):
                if modes and mode not in modes:
                    continue
                trace = serve.poisson_trace(rate, window, seed=seed)
                res = srv.serve(kw, trace, keep_log=(timeline_at == (rate, seed) and mode == "nova_adaptive"))
                res.update({"mode": mode, "rate_req_s": rate, "seed": seed, "window_s": window,
                            "decode_cus": list(kw.get("decode_cus", (256, 256)))})
                runs.append(res)
                log(f"serve {mode:26s} rate {rate} seed {seed}: max E2E {res['max_e2e_s']:.3f} s, avg "
                    f"{res['avg_e2e_s']:.3f} s, avg TBT {res['avg_tbt_ms']:.1f} ms, decode batch "
                    f"{res['avg_decode_batch']:.2f}, vision wait {res['avg_queue_wait_s']:.3f} s (Eq. 6: "
                    f"{res['eq6_predicted_wait_s']})")
    summary = []
    for rate in rates:
        for mode in dict.fromkeys(r["mode"] for r in runs):
            rs = [r for r in runs if r["mode"] == mode and r["rate_req_s"] == rate]
            if not rs:
                continue
            row = {"mode": mode, "rate_req_s": rate, "seeds": len(rs), "requests": int(sum(r["requests"] for r in rs))}
            for k in ("max_e2e_s", "avg_e2e_s", "avg_ttft_s", "avg_tbt_ms", "avg_decode_batch", "throughput_req_s",
                      "avg_queue_wait_s"):
                v = np.array([r[k] for r in rs], float)
                row[k] = round(float(v.mean()), 4)
                row[k + "_std"] = round(float(v.std()), 4)
            # Eq. 6 over the pooled service times of all seeds
            t = np.array([r["mean_service_s"] for r in rs])
            t2 = np.array([r["mean_service2_s2"] for r in rs])
            w = sched.mg1_wait(rate, float(t.mean()), float(t2.mean()))
            row["eq6_predicted_wait_s"] = None if w == float("inf") else round(w, 4)
            row["utilization"] = round(rate * float(t.mean()), 3)
            summary.append(row)
        sl = [r for r in summary if r["rate_req_s"] == rate and r["mode"] in ("time_sliced_decode_first",
                                                                               "time_sliced_prefill_first")]
        if sl:
            best = min(sl, key=lambda r: r["max_e2e_s"])
            summary.append(dict(best, mode="time_sliced_best", chosen=best["mode"]))
    return {"adaptive_params": adaptive, "summary": summary, "runs": runs}




def measure_corun(nova, torch, st, srv):
    """Decode (batch 8) on P CUs beside the screenshot encode or a 3.6k-token prefill on the other
    256 - P, for P = 32..224: the co-run curves the Eq. 3 search consumes."""
    corun = []
    for other in ("encode", "prefill"):
        for p in [32, 64, 96, 128, 160, 192, 224]:
            s_d = nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(p, 0))
            so = nova.set_stage_partition(nova.STAGE_ENCODE if other == "encode" else nova.STAGE_PREFILL,
                                          nova.make_cu_mask(256 - p, p // 8))
            run_other = (lambda: srv.encode(so)) if other == "encode" else (lambda: srv.prefill(so))
            t_o = time_passes(torch, run_other, 1, so)
            t_d = time_passes(torch, lambda: st.decode(8, stream=s_d), 5, s_d)
            n_dec = max(4, int(t_o / max(t_d, 1e-3)) + 2)
            torch.cuda.synchronize()
            eo0, eo1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ed0, ed1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            eo0.record(so)
            run_other()
            eo1.record(so)
            ed0.record(s_d)
            for _ in range(n_dec):
                st.decode(8, stream=s_d)
            ed1.record(s_d)
            torch.cuda.synchronize()
            t_oc = eo0.elapsed_time(eo1)
            t_dc = ed0.elapsed_time(ed1) / n_dec
            corun.append({"pair": f"decode+{other}", "decode_cus": p, "other_cus": 256 - p,
                          f"{other}_ms_solo_on_partition": round(t_o, 3), f"{other}_ms_corun": round(t_oc, 3),
                          "decode_step_ms_solo_on_partition": round(t_d, 3), "decode_step_ms_corun": round(t_dc, 3)})
            log(f"co-run decode {p} / {other} {256 - p}: {other} {t_oc:.2f} ms (solo {t_o:.2f}), "
                f"decode step {t_dc:.3f} ms (solo {t_d:.3f})")
    return corun


# ----------------------------------------------------------------------------- linear co-run study
def linear_corun(nova, torch, synth, n_dec=2000, n_vis=200):
    """The two-linear experiment of Sec. 3.2.1 (its linear co-run table and the SM sweep) and the
    intra-CU variant of Sec. 3.2.3 on MI355X: the vision MLP up-projection at the screenshot shape
    (13416 x 1280 -> 5120) repeated n_vis times and the decode gate/up projection at batch 3
    (3 x 3584 -> 2 x 18944) repeated n_dec times, each alone, both at once on unrestricted streams,
    on complementary CU partitions, and as the low-footprint pair (128x128-tile GEMM + vector-ALU
    decode linear without LDS) sharing every CU.  Per-launch times come from HIP events on each
    stream; the makespan spans the first and last event of both."""
    full = [0xFFFFFFFF] * 8
    g = torch.Generator(device="cuda")
    g.manual_seed(17)
    xv = (torch.randn(13416, 1280, generator=g, device="cuda")).to(torch.bfloat16)
    wv = (torch.randn(5120, 1280, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    ov = torch.zeros(13416, 5120, dtype=torch.float32, device="cuda")
    xd = (torch.randn(3, 3584, generator=g, device="cuda")).to(torch.bfloat16)
    wd = (torch.randn(2 * 18944, 3584, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    od = torch.zeros(3, 2 * 18944, dtype=torch.float32, device="cuda")

    def run(vis_variant, dec_variant, vis_cus, dec_cus, nv, nd):
        sv = nova.set_stage_partition(nova.STAGE_ENCODE, full if vis_cus == 256 else nova.make_cu_mask(vis_cus, 256 // 8 - vis_cus // 8))
        sd = nova.set_stage_partition(nova.STAGE_DECODE, full if dec_cus == 256 else nova.make_cu_mask(dec_cus, 0))
        torch.cuda.synchronize()
        ev_v = [torch.cuda.Event(enable_timing=True) for _ in range(nv + 1)]
        ev_d = [torch.cuda.Event(enable_timing=True) for _ in range(nd + 1)]
        if nv:
            ev_v[0].record(sv)
        if nd:
            ev_d[0].record(sd)
        iv = idd = 0
        while iv < nv or idd < nd:          # enqueue both streams in proportion
            if idd < nd and (iv >= nv or idd * nv <= iv * nd):
                nova.linear(dec_variant, xd, wd, od, stream=sd)
                idd += 1
                ev_d[idd].record(sd)
            else:
                nova.linear(vis_variant, xv, wv, ov, stream=sv)
                iv += 1
                ev_v[iv].record(sv)
        torch.cuda.synchronize()
        out = {"vision_cus": vis_cus, "decode_cus": dec_cus}
        starts, ends = [], []
        for name, ev, n, flops in (("vision", ev_v, nv, 2.0 * 13416 * 1280 * 5120), ("decode", ev_d, nd, None)):
            if not n:
                continue
            t = np.array([a.elapsed_time(b) for a, b in zip(ev, ev[1:])])
            out[name] = {"launches": n, "total_ms": round(float(t.sum()), 2), "mean_us": round(float(t.mean()) * 1e3, 1),
                         "p50_us": round(float(np.percentile(t, 50)) * 1e3, 1),
                         "p99_us": round(float(np.percentile(t, 99)) * 1e3, 1),
                         "cv": round(float(t.std() / t.mean()), 3)}
            if flops:
                out[name]["tflops"] = round(flops / (t.mean() / 1e3) / 1e12, 1)
            else:
                out[name]["hbm_gbs"] = round(wd.numel() * 2 / (t.mean() / 1e3) / 1e9, 1)
            starts.append(ev[0])
            ends.append(ev[-1])
        out["makespan_ms"] = round(max(starts[0].elapsed_time(e) for e in ends), 2) if starts else 0.0
        return out

    res = {"workload": "vision fc1 13416x1280->5120 (x%d), decode gate/up 3x3584->37888 (x%d)" % (n_vis, n_dec)}
    for v in (nova.LINEAR_TILED, nova.LINEAR_TILED_SMALL):      # warm every kernel once
        nova.linear(v, xv, wv, ov)
    for v in (nova.LINEAR_THIN, nova.LINEAR_THIN_VALU):
        nova.linear(v, xd, wd, od)
    torch.cuda.synchronize()
    T, TS, D, DV = nova.LINEAR_TILED, nova.LINEAR_TILED_SMALL, nova.LINEAR_THIN, nova.LINEAR_THIN_VALU
    res["solo_vision"] = run(T, D, 256, 256, n_vis, 0)
    res["solo_decode"] = run(T, D, 256, 256, 0, n_dec)
    res["sequential_ms"] = round(res["solo_vision"]["makespan_ms"] + res["solo_decode"]["makespan_ms"], 2)
    res["corun_unpartitioned"] = run(T, D, 256, 256, n_vis, n_dec)
    res["corun_partitioned"] = [run(T, D, 256 - p, p, n_vis, n_dec) for p in (16, 32, 48, 64, 96, 128)]
    res["solo_vision_small_tiles"] = run(TS, DV, 256, 256, n_vis, 0)
    res["solo_decode_valu"] = run(TS, DV, 256, 256, 0, n_dec)
    res["sequential_low_footprint_ms"] = round(res["solo_vision_small_tiles"]["makespan_ms"] +
                                               res["solo_decode_valu"]["makespan_ms"], 2)
    res["corun_intra_cu"] = run(TS, DV, 256, 256, n_vis, n_dec)
    for key in ("corun_unpartitioned", "corun_intra_cu"):
        r = res[key]
        log(f"linear co-run {key}: makespan {r['makespan_ms']} ms (sequential {res['sequential_ms']} ms); vision "
            f"{r['vision']['mean_us']} us cv {r['vision']['cv']}, decode {r['decode']['mean_us']} us cv {r['decode']['cv']}")
    for r in res["corun_partitioned"]:
        log(f"linear co-run decode on {r['decode_cus']} CUs: makespan {r['makespan_ms']} ms; vision {r['vision']['mean_us']} us, "
            f"decode {r['decode']['mean_us']} us")
    return res


# ----------------------------------------------------------------------------- offload (Sec. 3.5)
def measure_offload(nova, torch, st, srv, slots=(2, 3, 4, 5)):
    """The encoder with its 32 layers in pinned host memory, streamed through K device slots (Eq. 7),
    against the resident encoder, on three encode workloads; plus the Eq. 8 bandwidth each would need
    to hide the copies, next to the measured pinned host-to-device rate."""
    lb, L = st.vit.layer_bytes, st.vc.layers
    host = torch.empty(st.vit.layers.numel(), dtype=torch.bfloat16, pin_memory=True)
    host.copy_(st.vit.layers)
    dev = torch.empty_like(st.vit.layers)
    stream = torch.cuda.current_stream()
    dev.copy_(host, non_blocking=True)
    h2d_ms = time_passes(torch, lambda: dev.copy_(host, non_blocking=True), 3, stream)
    del dev
    h2d_gbs = host.numel() * 2 / (h2d_ms / 1e3) / 1e9
    work = [("screenshot_1092x2408_b1", srv.vit, srv.pixels, srv.vis),
            ("image_1008x1008_b1", st.vit, st.pixels[:1], st.enc_out[:1]),
            ("image_1008x1008_b8", st.vit, st.pixels, st.enc_out)]
    def pass_times(fn, warm, reps):
        # back-to-back passes (so a pass's head copies overlap the previous pass's tail), one event
        # between each two
        for _ in range(warm):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            fn()
            ev[i + 1].record(stream)
        ev[-1].synchronize()
        return [a.elapsed_time(b) for a, b in zip(ev, ev[1:])]

    def per_pass(fn, warm=2, reps=5):
        # median and best, since a pass now and then runs long on this machine, resident ones too
        ts = sorted(pass_times(fn, warm, reps))
        return ts[len(ts) // 2], ts[0]

    rows = []
    for name, vit, px, out in work:
        t_res, t_res_min = per_pass(lambda: vit.encode(px, out=out))
        ref = out.clone()
        # Eq. 8: hiding every copy needs B >= (S / T) (L - K) / (L - 2), S the whole encoder's bytes
        row = {"workload": name, "resident_ms": round(t_res, 3), "resident_best_ms": round(t_res_min, 3),
               "resident_layer_mb": round(L * lb / 1e6, 1)}
        for K in slots:
            ov = nova.Vit(vit.cfg, None, blobs=(vit.embed, host, vit.head, lb), n_slots=K)
            if K == slots[0]:
                # the first passes of a freshly built ring, one by one (the warm-up anomaly)
                row["fresh_ring_passes_ms"] = [round(t, 3) for t in pass_times(lambda: ov.encode(px, out=out), 0, 8)]
            t_off, t_off_min = per_pass(lambda: ov.encode(px, out=out))
            same = bool(torch.equal(out, ref))
            need = (L * lb) / (t_res / 1e3) * (L - K) / (L - 2) / 1e9
            row[f"k{K}"] = {"ms": round(t_off, 3), "best_ms": round(t_off_min, 3),
                            "overhead_pct": round(100 * (t_off / t_res - 1), 1),
                            "slot_mb": round(K * lb / 1e6, 1), "eq8_needed_gbs": round(need, 1),
                            "bit_identical": same}
            torch.cuda.synchronize()
            del ov
        rows.append(row)
        log(f"offload {name}: resident {t_res:.2f} ms; " + ", ".join(
            f"K={K} {row[f'k{K}']['ms']:.2f} ms (+{row[f'k{K}']['overhead_pct']}%, Eq. 8 needs "
            f"{row[f'k{K}']['eq8_needed_gbs']} GB/s)" for K in slots))
    del host
    return {"h2d_pinned_gbs": round(h2d_gbs, 1), "layer_mb": round(lb / 1e6, 2), "layers": L, "runs": rows}


# ----------------------------------------------------------------------------- CPU baseline
def _host_info():
    """Threads the oracle's BLAS uses, the BLAS library, and the host CPU model."""
    threads, blas = os.cpu_count() or 1, "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = [p for p in threadpool_info() if p.get("user_api") == "blas"] or threadpool_info()
        if info:
            threads = max(p.get("num_threads", 1) for p in info)
            blas = ", ".join(sorted({f"{p.get('internal_api', '?')} {p.get('version', '')}".strip() for p in info}))
    except Exception:
        pass
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return int(threads), blas, model


def cpu_baseline(synth):
    """The oracle, as is (float64 NumPy), on bounded samples of each stage at the real shapes:
    * encode: one 1008x1008 image's patch embedding, 2 of the 32 encoder layers and the adapter,
      extrapolated to a full pass (the headline unit, patches/s);
    * prefill: one of the 28 decoder layers over the 1500-token prompt plus the LM head on a
      1/16 slice of the vocabulary, extrapolated to 28 layers and the full head (tok/s);
    * decode: one step of batch 1, 8 and 32 through one layer at a 1500-token context, and the
      head slice, extrapolated the same way (tok/s);
    * the tiny stack end to end (encode, 96-token prefill, 16 greedy decode steps)."""
    import dataclasses
    from oracle import vlm
    threads, blas, model = _host_info()
    out = {}
    # encode
    cfg = synth.VIT_1008
    names = ["patch.w", "patch.b", "pos", "merge.ln.g", "merge.ln.b", "merge.w", "merge.b"] + synth.vit_layer_names(0)
    w = synth.vit_weights(cfg, seed=0, names=names)
    img = synth.image(1, cfg.image_h, cfg.image_w, seed=1)[0]
    t0 = time.perf_counter()
    x = vlm.patch_embed(img, w, cfg)
    t_embed = time.perf_counter() - t0
    layers_timed = 2
    t0 = time.perf_counter()
    for _ in range(layers_timed):
        x = vlm.vit_layer(x, w, 0, cfg)
    t_layer = (time.perf_counter() - t0) / layers_timed
    t0 = time.perf_counter()
    vlm.merge_adapter(x, w, cfg)
    t_merge = time.perf_counter() - t0
    t_img = t_embed + cfg.layers * t_layer + t_merge
    del w, x
    # prefill and decode: one real-width layer, the LM head on a vocabulary slice
    lc = synth.LLM_28
    vs = lc.vocab // 16
    l1 = dataclasses.replace(lc, layers=1, vocab=vs)
    wl = synth.llm_weights(l1, seed=0)
    nv, nt = synth.LLM_VISION_TOKENS, synth.LLM_TEXT_TOKENS
    s = nv + nt
    xs = np.concatenate([synth.vision_embeds(nv, lc.hidden), wl["embed"][synth.text_ids(nt, vs)]], 0)
    t0 = time.perf_counter()
    h, _, _ = vlm.llm_layer_rows(xs, wl, 0, l1, np.arange(s))
    t_pre_layer = time.perf_counter() - t0
    t0 = time.perf_counter()
    vlm.lm_head(h[-1:], wl, l1)
    t_head = (time.perf_counter() - t0) * (lc.vocab / vs)
    t_prefill = lc.layers * t_pre_layer + t_head
    tables, pool = synth.block_tables([s + 1], lc.block, seed=5)
    kv = vlm.PagedKV(1, pool, lc.n_kv, lc.block, lc.head_dim)
    rng = np.random.default_rng(0)
    kv.k[:] = rng.standard_normal(kv.k.shape)
    kv.v[:] = rng.standard_normal(kv.v.shape)
    t0 = time.perf_counter()
    vlm.llm_decode_step(np.array([5]), np.array([s]), tables, kv, wl, l1)
    t_dec1 = time.perf_counter() - t0
    t_decode = lc.layers * t_dec1 + t_head          # the slice's head time is inside t_dec1; upper bound
    del kv
    # batches of 8 and 32 sequences at the same context, the same way (head on B rows, scaled up)
    t_dec_b = {}
    for bsz in (8, 32):
        tb, pb = synth.block_tables([s + 1] * bsz, lc.block, seed=5)
        kvb = vlm.PagedKV(1, pb, lc.n_kv, lc.block, lc.head_dim)
        kvb.k[:] = rng.standard_normal(kvb.k.shape)
        kvb.v[:] = rng.standard_normal(kvb.v.shape)
        t0 = time.perf_counter()
        vlm.llm_decode_step(np.full(bsz, 5), np.full(bsz, s), tb, kvb, wl, l1)
        t_step = time.perf_counter() - t0
        t0 = time.perf_counter()
        vlm.lm_head(np.repeat(h[-1:], bsz, 0), wl, l1)
        t_dec_b[bsz] = lc.layers * t_step + (time.perf_counter() - t0) * (lc.vocab / vs)
        del kvb
    del wl
    # tiny stack end to end
    tv, tl = synth.TINY_VIT, synth.TINY_LLM
    wv, wt = synth.vit_weights(tv, 0), synth.llm_weights(tl, 0)
    timg = synth.image(1, tv.image_h, tv.image_w, seed=1)[0]
    tids = synth.text_ids(synth.TINY_TEXT, tl.vocab, seed=2)
    t0 = time.perf_counter()
    vis = vlm.vit_encode(timg, wv, tv)
    ts = vis.shape[0] + synth.TINY_TEXT
    ttab, tpool = synth.block_tables([ts + synth.TINY_DECODE_STEPS], tl.block, seed=5)
    tkv = vlm.PagedKV(tl.layers, tpool, tl.n_kv, tl.block, tl.head_dim)
    _, tok = vlm.llm_prefill(vis, tids, wt, tl, kv=tkv, table=ttab[0])
    for t in range(synth.TINY_DECODE_STEPS):
        tok = int(vlm.llm_decode_step(np.array([tok]), np.array([ts + t]), ttab, tkv, wt, tl)[1][0])
    t_tiny = time.perf_counter() - t0
    return {"value": round(cfg.n_patches / t_img, 2), "unit": "patches/s", "cores": threads, "kind": "oracle",
            "precision": "float64", "blas": blas, "cpu_model": model,
            "sample": f"1 image of {cfg.image_h}x{cfg.image_w} ({cfg.n_patches} patches): patch embed, "
                      f"{layers_timed} of {cfg.layers} encoder layers timed (float64 NumPy), adapter; "
                      f"full pass extrapolated as embed + {cfg.layers} x layer + adapter = {t_img:.1f} s",
            "stages": {"encode_image_s": round(t_img, 2),
                       "prefill_s1500_s": round(t_prefill, 2), "prefill_tok_per_s": round(s / t_prefill, 2),
                       "decode_b1_step_s": round(t_decode, 3), "decode_b1_tok_per_s": round(1 / t_decode, 3),
                       "decode_b8_step_s": round(t_dec_b[8], 3), "decode_b8_tok_per_s": round(8 / t_dec_b[8], 3),
                       "decode_b32_step_s": round(t_dec_b[32], 3), "decode_b32_tok_per_s": round(32 / t_dec_b[32], 3),
                       "tiny_stack_end_to_end_s": round(t_tiny, 3),
                       "note": "prefill and decode: 1 of 28 layers timed and the LM head on 1/16 of the "
                               "vocabulary, extrapolated to 28 layers and the full head"}}


# ----------------------------------------------------------------------------- main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--batch", type=int, default=8, help="images per encode pass (headline)")
    ap.add_argument("--no-sweep", action="store_true", help="skip CU-share curves and co-run")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--rates", type=float, nargs="+", default=[2.0, 4.0], help="request rates (req/s) of the serving runs")
    ap.add_argument("--window", type=float, default=10.0, help="arrival window (s) of each serving run")
    ap.add_argument("--seeds", type=int, nargs="+", default=[3], help="trace seeds of the serving runs")
    ap.add_argument("--serving-sweep", action="store_true",
                    help="only the co-run curves and the serving runs over --rates x --seeds (prints their JSON)")
    ap.add_argument("--hbm-budget", action="store_true",
                    help="only the serving runs under an HBM budget: encoder layers offloaded (K = 2 slots), "
                         "KV pool capped at 40 GB, batch-32 decode (prints their JSON)")
    ap.add_argument("--modes", nargs="+", default=None, help="restrict the serving modes")
    ap.add_argument("--linear-corun", action="store_true",
                    help="only the two-linear co-run study (inter-CU partitions vs intra-CU sharing; prints its JSON)")
    ap.add_argument("--only-encode", action="store_true", help="headline encode loop only (for profiling)")
    ap.add_argument("--profile-stage", choices=["prefill", "encode1", "decode1", "decode8", "decode32", "copy", "offload",
                                                "screenshot", "prefill_screenshot"],
                    help="run only this stage in a loop of --steps passes (for rocprofv3); 'copy' is a plain "
                         "1 GiB device copy that calibrates the HBM byte counters; 'offload' runs only the "
                         "layer-offload comparison; 'screenshot' and 'prefill_screenshot' are the serving shapes "
                         "(a 1092x2408 image, 13,416 patches; its 3354 visual tokens + 225 text tokens)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the method serves all three stages on a single GPU; "
              "multi-GPU runs are not supported (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2509_21301_amd import nova, sched, serve, synth
    device = "cuda"
    if args.profile_stage == "copy":
        src = torch.ones(1 << 30, dtype=torch.uint8, device=device)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        ms = time_passes(torch, lambda: dst.copy_(src), args.steps, torch.cuda.current_stream())
        log(f"copy 1 GiB: {ms:.3f} ms per pass, {2 * (1 << 30) / (ms / 1e3) / 1e9:.1f} GB/s (read + write)")
        return
    nova.init(0)
    if args.linear_corun:
        print(json.dumps({"linear_corun": linear_corun(nova, torch, synth)}), flush=True)
        return
    st = Stages(nova, torch, synth, device, args.batch)
    vc, lc = st.vc, st.lc
    B = args.batch
    stream = torch.cuda.current_stream()

    if args.serving_sweep or args.hbm_budget:
        out_len = 32.0
        srv = ServingSetup(nova, torch, synth, st)
        corun = measure_corun(nova, torch, st, srv)
        curves = sched.StageCurves.from_corun(corun)
        res = {"corun": corun}
        if args.serving_sweep:
            sv = run_serving(serve, sched, srv, curves, out_len, args.rates, args.seeds, args.window, modes=args.modes,
                             timeline_at=(args.rates[-1], args.seeds[0]))
            res["serving_sweep"] = sv
        if args.hbm_budget:
            # Sec. 3.5 inside serving: 40 GB of KV blocks (43,596 of 917,504 bytes), the encoder's 32
            # layers streamed through 2 device slots, requests at --rates with decode batches up to 32
            kv_blocks = int(40e9 // (lc.layers * 2 * lc.n_kv * lc.block * lc.head_dim * 2))
            del srv
            torch.cuda.empty_cache()
            off = ServingSetup(nova, torch, synth, st, n_slots=2, kv_blocks=kv_blocks)
            sv = run_serving(serve, sched, off, curves, out_len, args.rates, args.seeds, args.window, modes=args.modes)
            sv["kv_blocks"], sv["kv_gb"] = kv_blocks, round(off.kv.k.numel() * 4 / 1e9, 2)
            sv["encoder_device_mb"] = round(2 * st.vit.layer_bytes / 1e6, 1)
            res["hbm_budget"] = sv
            # the same traces with the encoder resident, for the offload overhead inside serving
            del off
            torch.cuda.empty_cache()
            res_srv = ServingSetup(nova, torch, synth, st, kv_blocks=kv_blocks)
            res["hbm_budget_resident_encoder"] = run_serving(
                serve, sched, res_srv, curves, out_len, args.rates, args.seeds, args.window,
                modes=["nova_adaptive", "nova_rate_static"])
        print(json.dumps(res), flush=True)
        return

    if args.profile_stage == "offload":
        print(json.dumps(measure_offload(nova, torch, st, ServingSetup(nova, torch, synth, st))), flush=True)
        return
    if args.profile_stage in ("screenshot", "prefill_screenshot"):
        srv = ServingSetup(nova, torch, synth, st)
        srv.encode(stream)                 # the prefill's visual tokens
        fn = (lambda: srv.encode(stream)) if args.profile_stage == "screenshot" else (lambda: srv.prefill(stream))
        for _ in range(args.warmup):
            fn()
        ms = time_passes(torch, fn, args.steps, stream)
        log(f"{args.profile_stage}: {ms:.3f} ms per pass")
        return
    if args.profile_stage:
        fn = {"prefill": st.prefill, "encode1": lambda: st.encode(1)}.get(
            args.profile_stage, lambda: st.decode(int(args.profile_stage[6:])))
        for _ in range(args.warmup):
            fn()
        ms = time_passes(torch, fn, args.steps, stream)
        log(f"{args.profile_stage}: {ms:.3f} ms per pass")
        return

    # ---------------- headline: encode, batch B, all CUs (no per-kernel events in the timed loop)
    for _ in range(args.warmup):
        st.encode()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        st.encode()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1)
    ms_step = ms / args.steps
    value = B * vc.n_patches * args.steps / (ms / 1e3)
    gemm_f, attn_f = vit_flops(vc, B)
    log(f"encode batch {B}: {ms_step:.2f} ms/pass, {value:.0f} patches/s, "
        f"{(gemm_f + attn_f) / (ms_step / 1e3) / 1e12:.1f} TFLOP/s overall (wall {wall:.2f}s)")
    # kernel families: the same passes again with every family launch bracketed by HIP events that
    # the library records on the stream it launches on
    fam_steps = max(2, args.steps // 2)
    nova.timing_enable(True)
    for k in nova.KIND_NAMES:
        nova.timing_read(k)
    for _ in range(fam_steps):
        st.encode()
    torch.cuda.synchronize()
    kinds = {nova.KIND_NAMES[k]: nova.timing_read(k) for k in nova.KIND_NAMES}
    nova.timing_enable(False)
    for nm, (t, n) in kinds.items():
        log(f"  {nm:18s} {t / fam_steps:9.3f} ms/pass  {n / fam_steps:6.1f} launches/pass")
    # dominant kernel family of the pass and its roofline position
    fam_flops = {"gemm": gemm_f, "attention": attn_f}
    dom = max(fam_flops, key=lambda f: kinds[f][0])
    t_dom, n_dom = kinds[dom]
    flops_per_launch = fam_flops[dom] * fam_steps / max(n_dom, 1)
    achieved = flops_per_launch / ((t_dom / max(n_dom, 1)) / 1e3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                "traffic": gemm_traffic() if dom == "gemm" else None,
                "avg_launch_ms": round(t_dom / max(n_dom, 1), 4),
                "flops_per_launch": flops_per_launch,
                "family_passes": fam_steps,
                "family_ms_per_pass": {f: round(kinds[f][0] / fam_steps, 3) for f in kinds},
                "other_kernels": {f: round(fam_flops[f] * fam_steps / kinds[f][0] / 1e9, 1)
                                  for f in fam_flops if f != dom and kinds[f][0] > 0}}

    result = {
        "metric": "per-stage tok/s and patches/s vs CU share; co-run max latency at 1 GPU",
        "value": round(value, 1), "unit": "patches/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded uniform-noise images, random N(0,0.02) bf16 weights)",
        "config": {"workload": f"vision encode, ViT 32x1280 (16 heads, MLP 5120, patch 14, 2x2 merge to 3584), "
                               f"{B} images of {vc.image_h}x{vc.image_w} ({vc.n_patches} patches each) per step",
                   "global_batch": B, "seq_len": vc.n_patches, "parallelism": "single GPU, 256 CUs"},
        "roofline": roofline,
    }
    if args.only_encode:
        print(json.dumps(result), flush=True)
        return

    # ---------------- per-stage throughput on all CUs: median (p10, p90) of per-pass event times,
    # rates and roofline fractions at the median (useful flops only; decode against HBM bytes)
    stages = {}
    for b in (1, 4, 8):
        if b > B:
            continue
        st.encode(b)
        sp = spread(time_each(torch, lambda: st.encode(b), 10, stream))
        t = sp["ms"]
        tf = sum(vit_flops(vc, b)) / (t / 1e3) / 1e12
        stages[f"encode_b{b}"] = {**sp, "patches_per_s": round(b * vc.n_patches / (t / 1e3), 1),
                                  "tflops": round(tf, 1), "frac": round(tf / BF16_PEAK_TFLOPS, 3)}
    st.prefill()
    sp = spread(time_each(torch, st.prefill, 20, stream))
    t = sp["ms"]
    pf_lin, pf_attn = prefill_flops(lc, st.s)
    tf = (pf_lin + pf_attn) / (t / 1e3) / 1e12
    stages["prefill_s1500"] = {**sp, "tok_per_s": round(st.s / (t / 1e3), 1), "tflops": round(tf, 1),
                               "frac": round(tf / BF16_PEAK_TFLOPS, 3)}
    for b in (1, 8, 32):
        st.decode(b)
        sp = spread(time_each(torch, lambda: st.decode(b), 30, stream))
        t = sp["ms"]
        wb, kvb = decode_bytes(lc, b, st.s + 1)          # every sequence sits at position s: s + 1 keys
        stages[f"decode_b{b}"] = {**sp, "tok_per_s": round(b / (t / 1e3), 1),
                                  "hbm_gbs": round((wb + kvb) / (t / 1e3) / 1e9, 1),
                                  "hbm_frac": round((wb + kvb) / (t / 1e3) / 1e9 / HBM_PEAK_GBS, 3)}
    result["stages"] = stages
    log(json.dumps(stages))

    # ---------------- CU-share curves and co-run (XCD-balanced partitions)
    if not args.no_sweep:
        shares = [32, 64, 96, 128, 160, 192, 224, 256]
        curves = {"shares": shares, "encode_b1_patches_per_s": [], "prefill_tok_per_s": [], "decode_b8_tok_per_s": [],
                  # fractions of the full-GPU peak and of the share's own compute peak (P / 256 of it);
                  # decode against the full HBM bandwidth
                  "encode_b1_frac": [], "encode_b1_frac_of_share": [], "prefill_frac": [], "prefill_frac_of_share": [],
                  "decode_b8_hbm_frac": []}
        enc1_flops = sum(vit_flops(vc, 1))
        pf_flops = sum(prefill_flops(lc, st.s))
        dec8_bytes = sum(decode_bytes(lc, 8, st.s + 1))
        for p in shares:
            ms_e = ms_p = ms_d = None
            s_e = nova.set_stage_partition(nova.STAGE_ENCODE, nova.make_cu_mask(p, 0))
            ms_e = time_passes(torch, lambda: st.encode(1, stream=s_e), 2, s_e)
            s_p = nova.set_stage_partition(nova.STAGE_PREFILL, nova.make_cu_mask(p, 0))
            ms_p = time_passes(torch, lambda: st.prefill(stream=s_p), 2, s_p)
            s_d = nova.set_stage_partition(nova.STAGE_DECODE, nova.make_cu_mask(p, 0))
            ms_d = time_passes(torch, lambda: st.decode(8, stream=s_d), 5, s_d)
            curves["encode_b1_patches_per_s"].append(round(vc.n_patches / (ms_e / 1e3), 1))
            curves["prefill_tok_per_s"].append(round(st.s / (ms_p / 1e3), 1))
            curves["decode_b8_tok_per_s"].append(round(8 / (ms_d / 1e3), 1))
            fe = enc1_flops / (ms_e / 1e3) / 1e12 / BF16_PEAK_TFLOPS
            fp = pf_flops / (ms_p / 1e3) / 1e12 / BF16_PEAK_TFLOPS
            curves["encode_b1_frac"].append(round(fe, 3))
            curves["encode_b1_frac_of_share"].append(round(fe * 256 / p, 3))
            curves["prefill_frac"].append(round(fp, 3))
            curves["prefill_frac_of_share"].append(round(fp * 256 / p, 3))
            curves["decode_b8_hbm_frac"].append(round(dec8_bytes / (ms_d / 1e3) / 1e9 / HBM_PEAK_GBS, 3))
            log(f"share {p:3d} CUs: encode {ms_e:.2f} ms, prefill {ms_p:.2f} ms, decode(b8) {ms_d:.3f} ms")
        result["cu_share_curves"] = curves
        # co-run on the serving shapes: decode (batch 8) on P CUs with the screenshot encode or a
        # 3.5k-token prefill on the other 256 - P; these are the curves the Eq. 3 search consumes
        srv = ServingSetup(nova, torch, synth, st)
        corun = measure_corun(nova, torch, st, srv)
        result["corun"] = corun
        # offload: the Sec. 3.5 ring against the resident encoder, with the Eq. 8 bandwidth check
        result["offload"] = measure_offload(nova, torch, st, srv)
        curves = sched.StageCurves.from_corun(corun)
        out_len = 32.0                                   # mean of the U{16..48} output lengths
        pv, pp, lat = sched.best_static(curves, out_len)
        result["static_optimum"] = {"decode_cus_with_encode": pv, "decode_cus_with_prefill": pp,
                                    "expected_e2e_s": round(lat, 4), "mean_output_tokens": out_len,
                                    "ideal_req_per_s": round(sched.ideal_throughput(curves, pv, pp), 3)}
        result["pareto_front"] = [{"e2e_s": round(a, 4), "req_per_s": round(b, 3), "decode_cus_with_encode": c,
                                   "decode_cus_with_prefill": d} for a, b, c, d in sched.pareto_front(curves, out_len)]
        log(f"Eq. 3 optimum: decode {pv} CUs beside encode, {pp} beside prefill, expected E2E {lat:.3f} s")
        # serving: Poisson bursts through the Alg. 1 policy, co-run partitions vs time slicing
        result["rate_optimum"] = []
        for rate in args.rates:
            # the Pareto point for this rate: Eq. 1 plus the Eq. 6 queueing delay of encode + prefill
            rv, rp, rlat = sched.best_under_load(sched.on_granule(curves), out_len, rate)
            result["rate_optimum"].append({"rate_req_s": rate, "decode_cus_with_encode": rv,
                                           "decode_cus_with_prefill": rp, "expected_e2e_s": round(rlat, 4)})
        sv = run_serving(serve, sched, srv, curves, out_len, args.rates, args.seeds, args.window,
                         timeline_at=(args.rates[-1], args.seeds[0]))
        result["adaptive_params"] = {k: v for k, v in sv["adaptive_params"].items() if k != "points"}
        result["serving"] = sv["summary"]
        result["serving_runs"] = [{k: v for k, v in r.items() if k not in ("partition_timeline", "arrivals_ms")}
                                  for r in sv["runs"]]
        result["partition_timeline"] = next((dict(mode=r["mode"], rate_req_s=r["rate_req_s"], seed=r["seed"],
                                                  timeline=r["partition_timeline"], arrivals_ms=r["arrivals_ms"])
                                             for r in sv["runs"] if "partition_timeline" in r), None)

    if not args.no_cpu:
        log("timing the oracle on the host (bounded sample)")
        result["cpu_baseline"] = cpu_baseline(synth)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
