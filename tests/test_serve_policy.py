"""The Alg. 1 serving policy on the host, with the GPU passes replaced by timed stand-ins:
vision encode and prefill never overlap, prefill runs before the next vision pass, vision waits
in FIFO order, decode requests join the running batch at step boundaries and every request gets
exactly its n_out tokens; the time-sliced driver runs one pass at a time."""
import threading
import time
from types import SimpleNamespace

import pytest

from paper_2509_21301_amd import serve, synth


def fake_server(mode, **kw):
    cfg = synth.TINY_LLM
    vit = SimpleNamespace(cfg=SimpleNamespace(n_out=64))
    llm = SimpleNamespace(cfg=cfg)
    kv = SimpleNamespace(num_blocks=2000)
    srv = serve.Server(vit, llm, kv, None, mode=mode, max_batch=4, max_blocks=64, device="cpu", **kw)
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
        pos, max_ctx = srv._decode_positions(batch)      # what the real step hands the library
        span("decode", 0.003)
        now = time.perf_counter()
        for r, p in zip(batch, pos):
            r.t_tokens.append(now)
            srv.fed_positions.setdefault(r.rid, []).append((p, max_ctx))
        log.append(("decode", tuple(r.rid for r in batch)))

    srv._vision, srv._prefill, srv._decode_step = vision, prefill, decode
    srv.fed_positions = {}
    return srv, log


SLICED = {"sliced_alternate": dict(slice_order="alternate"), "sliced_decode_first": dict(slice_order="decode_first"),
          "sliced_prefill_first": dict(slice_order="prefill_first"),
          "pf_limit": dict(slice_order="prefill_first", decode_limit=5)}


@pytest.mark.parametrize("mode", ["nova", *SLICED])
def test_alg1_policy(mode):
    srv, log = fake_server("nova" if mode == "nova" else "time_sliced", **SLICED.get(mode, {}))
    trace = serve.poisson_trace(rate=200.0, window_s=0.08, seed=1, n_text=(5, 9), n_out=(6, 12))
    assert len(trace) >= 8
    res = srv.run(trace)
    assert res["requests"] == len(trace)
    for r in trace:
        assert len(r.t_tokens) == r.n_out
        assert r.t_arrive <= r.t_vis0 <= r.t_vis1 <= r.t_pre1 <= r.t_tokens[0]
    starts = [e[2] for e in log if e[0] == "start"]
    assert all(a["vision"] + a["prefill"] <= 1 for a in starts)          # never vision with prefill
    if mode != "nova":
        assert all(a["any"] <= 1 for a in starts)                        # one pass at a time
    order = [e for e in log if e[0] in ("vision", "prefill")]
    vis = [e[1] for e in order if e[0] == "vision"]
    assert vis == sorted(vis)                                            # FIFO vision queue
    for i, e in enumerate(order):                                        # prefill right after its vision
        if e[0] == "vision":
            assert order[i + 1] == ("prefill", e[1])
    batches = [e[1] for e in log if e[0] == "decode"]
    if mode != "sliced_decode_first":     # decode-first finishes each batch before the next prefill
        assert max(len(b) for b in batches) > 1                          # in-flight batching happened
    # decode step t of a request feeds token t at position S + t (prefill wrote 0..S-1 and emitted
    # token 0), and the step's max_ctx covers every sequence of the batch
    for r in trace:
        s_len = 64 + r.n_text
        fed = srv.fed_positions[r.rid]
        assert [p for p, _ in fed] == list(range(s_len, s_len + r.n_out - 1)), r.rid
        assert all(p < m for p, m in fed)
        assert (s_len + r.n_out - 2) // 16 < len(r.blocks)                 # the last fed position has a block
    assert srv.blocks.free and len(srv.blocks.free) == 2000             # every KV block returned
    assert res["max_e2e_s"] >= res["avg_e2e_s"] > 0
    # statistics: decode batch sizes of every step, Eq. 6 beside the measured vision-queue wait
    assert res["decode_steps"] == len(batches)
    assert abs(res["avg_decode_batch"] - sum(len(b) for b in batches) / len(batches)) < 1e-3
    assert res["mean_service_s"] > 0 and "eq6_predicted_wait_s" in res
    if mode == "nova":
        assert res["sched_event_us"]["n"] >= 2 * len(trace)
        assert res["sched_event_us"]["p10"] <= res["sched_event_us"]["p50"] <= res["sched_event_us"]["p99"]


def test_decode_positions_after_prefill():
    srv, _ = fake_server("nova")
    a = serve.Request(0, 0.0, n_text=10, n_out=5)
    b = serve.Request(1, 0.0, n_text=30, n_out=5)
    a.t_tokens = [0.1]                  # just prefilled: feeds token 0 at S = 64 + 10
    b.t_tokens = [0.1, 0.2, 0.3]        # two decode steps done: feeds token 2 at S + 2
    pos, max_ctx = srv._decode_positions([a, b])
    assert pos == [74, 96] and max_ctx == 97


@pytest.mark.parametrize("order,limit,n_batch,n_decode,other,last,want", [
    ("alternate", None, 2, 2, True, False, True), ("alternate", None, 2, 2, True, True, False),
    ("alternate", None, 0, 0, True, False, False), ("decode_first", None, 1, 1, True, True, True),
    ("prefill_first", None, 3, 9, True, False, False), ("prefill_first", None, 3, 3, False, True, True),
    ("prefill_first", 5, 4, 5, True, False, False), ("prefill_first", 5, 4, 6, True, True, True)])
def test_time_sliced_orders(order, limit, n_batch, n_decode, other, last, want):
    srv, _ = fake_server("time_sliced", slice_order=order, decode_limit=limit)
    assert srv._slice_decode_next(n_batch, n_decode, other, last) is want


def test_worker_error_ends_the_run():
    srv, _ = fake_server("nova")

    def broken(req):
        raise RuntimeError("launch failed")
    srv._vision = broken
    trace = serve.poisson_trace(rate=200.0, window_s=0.05, seed=2, n_text=(5, 9), n_out=(6, 12))
    t0 = time.perf_counter()
    with pytest.raises(RuntimeError, match="serving worker failed"):
        srv.run(trace)
    assert time.perf_counter() - t0 < 10


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


@pytest.mark.parametrize("mode", ["nova", "time_sliced"])
def test_kv_blocks_taken_at_admission(mode):
    """KV blocks are taken when a request starts vision encode and returned when it finishes: with
    a pool that holds two requests at a time, a burst still completes, never holding more."""
    srv, _ = fake_server(mode)
    trace = serve.poisson_trace(rate=300.0, window_s=0.05, seed=4, n_text=(5, 9), n_out=(6, 12))
    need = max(srv._blocks_needed(r) for r in trace)
    srv.blocks = serve.BlockPool(2 * need)
    srv.kv.num_blocks = 2 * need
    seen = []
    take = srv.blocks.try_take

    def watched(n):
        got = take(n)
        seen.append(len(srv.blocks.free))
        return got
    srv.blocks.try_take = watched
    res = srv.run(trace)
    assert res["requests"] == len(trace) >= 6
    assert all(len(r.t_tokens) == r.n_out for r in trace)
    assert min(seen) >= 0 and len(srv.blocks.free) == 2 * need
