"""The Alg. 1 serving policy on the host, with the GPU passes replaced by timed stand-ins:
vision encode and prefill never overlap, prefill runs before the next vision pass, vision waits
in FIFO order, decode requests join the running batch at step boundaries and every request gets
exactly its n_out tokens; the time-sliced driver runs one pass at a time."""
import threading
import time
from types import SimpleNamespace

import pytest

from paper_2509_21301_amd import serve, synth


def fake_server(mode):
    cfg = synth.TINY_LLM
    vit = SimpleNamespace(cfg=SimpleNamespace(n_out=64))
    llm = SimpleNamespace(cfg=cfg)
    kv = SimpleNamespace(num_blocks=2000)
    srv = serve.Server(vit, llm, kv, None, mode=mode, max_batch=4, max_blocks=64, device="cpu")
    log, lock = [], threading.Lock()
    active = {"vision": 0, "prefill": 0, "decode": 0, "any": 0}

    def span(kind, dur, fn=None):
        with lock:
            active[kind] += 1
            active["any"] += 1
            log.append(("start", kind, dict(active)))
        time.sleep(dur)
        if fn:
            fn()
        with lock:
            active[kind] -= 1
            active["any"] -= 1

    def vision(req):
        req.t_vis0 = time.perf_counter()
        span("vision", 0.004)
        req.t_vis1 = time.perf_counter()
        log.append(("vision", req.rid))

    def prefill(req):
        span("prefill", 0.003)
        req.last_token = 1
        req.t_pre1 = time.perf_counter()
        log.append(("prefill", req.rid))

    def decode(batch):
        assert len(batch) <= 4
        span("decode", 0.003)
        now = time.perf_counter()
        for r in batch:
            r.t_tokens.append(now)
        log.append(("decode", tuple(r.rid for r in batch)))

    srv._vision, srv._prefill, srv._decode_step = vision, prefill, decode
    return srv, log


@pytest.mark.parametrize("mode", ["nova", "time_sliced"])
def test_alg1_policy(mode):
    srv, log = fake_server(mode)
    trace = serve.poisson_trace(rate=200.0, window_s=0.08, seed=1, n_text=(5, 9), n_out=(6, 12))
    assert len(trace) >= 8
    res = srv.run(trace)
    assert res["requests"] == len(trace)
    for r in trace:
        assert len(r.t_tokens) == r.n_out
        assert r.t_arrive <= r.t_vis0 <= r.t_vis1 <= r.t_pre1 <= r.t_tokens[0]
    starts = [e[2] for e in log if e[0] == "start"]
    assert all(a["vision"] + a["prefill"] <= 1 for a in starts)          # never vision with prefill
    if mode == "time_sliced":
        assert all(a["any"] <= 1 for a in starts)                        # one pass at a time
    order = [e for e in log if e[0] in ("vision", "prefill")]
    vis = [e[1] for e in order if e[0] == "vision"]
    assert vis == sorted(vis)                                            # FIFO vision queue
    for i, e in enumerate(order):                                        # prefill right after its vision
        if e[0] == "vision":
            assert order[i + 1] == ("prefill", e[1])
    batches = [e[1] for e in log if e[0] == "decode"]
    assert max(len(b) for b in batches) > 1                              # in-flight batching happened
    assert srv.blocks.free and len(srv.blocks.free) == 2000             # every KV block returned
    assert res["max_e2e_s"] >= res["avg_e2e_s"] > 0
    # statistics: decode batch sizes of every step, Eq. 6 beside the measured vision-queue wait
    assert res["decode_steps"] == len(batches)
    assert abs(res["avg_decode_batch"] - sum(len(b) for b in batches) / len(batches)) < 1e-3
    assert res["mean_service_s"] > 0 and "eq6_predicted_wait_s" in res
    if mode == "nova":
        assert res["sched_event_us"]["events"] >= 2 * len(trace)


def test_block_pool_exhaustion_is_an_error():
    p = serve.BlockPool(3)
    a = p.take(2)
    with pytest.raises(Exception):
        p.take(2)
    p.give(a)
    assert len(p.take(3)) == 3


def test_poisson_trace_is_seeded_and_bounded():
    a = serve.poisson_trace(2.0, 10.0, seed=3)
    b = serve.poisson_trace(2.0, 10.0, seed=3)
    assert [r.arrival for r in a] == [r.arrival for r in b]
    assert all(0 < r.arrival < 10 for r in a) and 8 <= len(a) <= 40
    assert all(150 <= r.n_text <= 300 and 16 <= r.n_out <= 48 for r in a)
