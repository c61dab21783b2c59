"""Co-run serving driver: requests (screenshot + instruction) flow through vision encode,
prefill and in-flight-batched decode on one GPU, scheduled by the policy of the paper's Alg. 1.

Policy (Sec. 3.4): FIFO within a stage; decode has the highest priority and co-runs with vision
encode or prefill on disjoint CU partitions; vision encode and prefill never run together, and
prefill goes before vision; decode requests join the running batch at the next step (in-flight
batching); partitions change only at forward-pass boundaries.  Partition modes:

* ``nova``         -- decode holds P CUs while co-running, the other stage 256 - P (static P,
                      or Eq. 5 from the number of requests in vision/prefill);
* ``multi_stream`` -- the same worker threads on unrestricted streams (the paper's Multi-Stream);
* ``time_sliced``  -- one worker runs one forward pass at a time on the whole GPU, in one of three
                      orders: a decode step between encode/prefill passes, decode first, or
                      encode/prefill first (optionally with the PF-Limit decode threshold of the
                      paper's Sec. 5.1 baselines).

Every worker is a thread that enqueues its pass on its stream through the C ABI and waits for
it; the scheduler thread owns the request state.  All timing is wall clock.
"""
from __future__ import annotations

import queue
import threading
import time
from dataclasses import dataclass, field

import numpy as np
import torch

from . import nova, sched, synth

FULL = [0xFFFFFFFF] * 8


@dataclass
class Request:
    rid: int
    arrival: float                 # seconds after the trace start
    n_text: int
    n_out: int
    ids: torch.Tensor = None
    table_row: np.ndarray = None
    blocks: list = field(default_factory=list)
    t_arrive: float = 0.0
    t_vis0: float = 0.0
    t_vis1: float = 0.0
    t_pre1: float = 0.0
    t_tokens: list = field(default_factory=list)
    last_token: int = 0

    @property
    def done(self):
        return len(self.t_tokens) >= self.n_out


def poisson_trace(rate, window_s, seed, n_text=(150, 300), n_out=(16, 48)):
    """Poisson(rate) arrivals over one window; text length and output length uniform (inclusive)."""
    r = np.random.default_rng([seed, int(rate * 1000)])
    t, out = 0.0, []
    while True:
        t += r.exponential(1.0 / rate)
        if t >= window_s:
            break
        out.append(Request(len(out), t, int(r.integers(n_text[0], n_text[1] + 1)), int(r.integers(n_out[0], n_out[1] + 1))))
    return out


class BlockPool:
    """Host free list of paged-KV blocks."""

    def __init__(self, n):
        self.free = list(range(n))[::-1]
        self.lock = threading.Lock()

    def take(self, n):
        with self.lock:
            if len(self.free) < n:
                raise nova.NovaError(nova.ENOKV, f"KV pool exhausted ({n} blocks wanted, {len(self.free)} free)")
            return [self.free.pop() for _ in range(n)]

    def try_take(self, n):
        """n blocks, or None (nothing taken) when fewer are free."""
        with self.lock:
            if len(self.free) < n:
                return None
            return [self.free.pop() for _ in range(n)]

    def available(self):
        with self.lock:
            return len(self.free)

    def give(self, blocks):
        with self.lock:
            self.free.extend(blocks)


class Server:
    def __init__(self, vit, llm, kv, pixels, mode="nova", decode_cus=(96, 96), alpha=0, minimum=32, max_batch=32,
                 max_blocks=256, device="cuda", slice_order="alternate", decode_limit=None, granule=sched.GRANULE):
        """decode_cus = (P_v, P_p): decode's CUs while co-running with vision encode / prefill
        (Eq. 3's optimum); alpha > 0 (one value, or one per pair as (alpha_v, alpha_p)) turns on
        the Eq. 5 adaptation with floor `minimum`, its shares rounded down to `granule` CUs.
        slice_order / decode_limit choose the time-sliced driver's pass order (see
        _slice_decode_next)."""
        if slice_order not in ("alternate", "decode_first", "prefill_first"):
            raise ValueError(f"unknown slice_order {slice_order!r}")
        self.vit, self.llm, self.kv, self.pixels, self.device = vit, llm, kv, pixels, device
        self.mode, self.decode_cus, self.alpha, self.minimum, self.granule = mode, decode_cus, alpha, minimum, granule
        self.slice_order, self.decode_limit = slice_order, decode_limit
        self.other = None             # stage co-running with decode: STAGE_ENCODE, STAGE_PREFILL or None
        self.max_batch, self.max_blocks = max_batch, max_blocks
        self.cfg = llm.cfg
        self.blocks = BlockPool(kv.num_blocks)
        self.n_vis = vit.cfg.n_out
        self.vis_buf = torch.empty(1, self.n_vis, self.cfg.hidden, dtype=torch.bfloat16, device=device)
        self.events = queue.Queue()
        self.lock = threading.Lock()
        self.n_pending = 0            # requests queued for or inside vision encode / prefill
        self.decode_active = 0        # requests in the decode batch or waiting to join it
        reserve = getattr(llm, "reserve", None)
        if reserve is not None:       # workspaces sized once, before any timed pass
            reserve(prefill_tokens=max_blocks * self.cfg.block, decode_batch=max_batch,
                    decode_ctx=max_blocks * self.cfg.block)
        self.partition_log = []
        self.decode_batches = []      # batch size of every decode step
        self.sched_us = []            # scheduler time per handled event (host, microseconds)
        self.worker_us = []           # worker time per pass to pick and switch its partition (host, us)

    # ---------------------------------------------------------------- partitions
    def _masks(self, stage):
        """Mask for `stage` at a pass boundary, from the current load (Eq. 5 when alpha > 0)."""
        if self.mode != "nova":
            return FULL
        with self.lock:
            pend, dec, other = self.n_pending, self.decode_active, self.other
        if stage == nova.STAGE_DECODE and other is None:
            return FULL
        if stage != nova.STAGE_DECODE and dec == 0:
            return FULL
        pair = stage if stage != nova.STAGE_DECODE else other
        i = 0 if pair == nova.STAGE_ENCODE else 1
        op = self.decode_cus[i]
        alpha = self.alpha[i] if isinstance(self.alpha, (tuple, list)) else self.alpha
        p = sched.decode_cus(pend, op, alpha, self.minimum, self.granule) if alpha else op
        return nova.make_cu_mask(p, 0) if stage == nova.STAGE_DECODE else nova.make_cu_mask(256 - p, p // 8)

    def _stream(self, stage):
        """The stream for the next forward pass of `stage` (the worker-side partition step, once
        per pass; its host time is the worker overhead of Sec. 5.7)."""
        if self.mode == "time_sliced":
            return torch.cuda.current_stream()
        t0 = time.perf_counter()
        mask = self._masks(stage)
        s = nova.set_stage_partition(stage, mask)
        t1 = time.perf_counter()
        self.worker_us.append((t1 - t0) * 1e6)
        self.partition_log.append((t1, stage, sum(bin(w).count("1") for w in mask)))
        return s

    # ---------------------------------------------------------------- stage passes
    def _vision(self, req):
        s = self._stream(nova.STAGE_ENCODE)
        req.t_vis0 = time.perf_counter()
        self.vit.encode(self.pixels, out=self.vis_buf, stream=s)
        s.synchronize()
        req.t_vis1 = time.perf_counter()

    # Host <-> device copies go on the stage's own stream: torch's default stream is HIP's null
    # stream, which waits for every other (blocking) stream, so a copy there would hold one
    # stage until the co-running stage's pass ends.
    def _prefill(self, req):
        s = self._stream(nova.STAGE_PREFILL)
        with torch.cuda.stream(s):
            tbl = torch.from_numpy(req.table_row).to("cuda", non_blocking=False)
            nxt = self.llm.prefill(self.vis_buf[0], req.ids, tbl, self.kv, stream=s)
            s.synchronize()
            req.last_token = int(nxt.item())
        req.t_pre1 = time.perf_counter()

    def _decode_positions(self, batch):
        """Position of the token each request feeds in its next decode step, and the step's max_ctx.

        Prefill writes positions 0..S-1 (S = visual + text tokens) and emits token 0; decode step
        t feeds token t at position S + t, so a request that holds k generated tokens feeds its
        last one at S + k - 1 and attends to S + k keys."""
        pos = [self.n_vis + r.n_text + len(r.t_tokens) - 1 for r in batch]
        return pos, max(pos) + 1

    def _decode_step(self, batch):
        s = self._stream(nova.STAGE_DECODE)
        ids = torch.tensor([r.last_token for r in batch], dtype=torch.int32)
        pos_l, max_ctx = self._decode_positions(batch)
        pos = torch.tensor(pos_l, dtype=torch.int32)
        tab = torch.from_numpy(np.stack([r.table_row for r in batch]))
        with torch.cuda.stream(s):
            ids_d, pos_d, tab_d = ids.cuda(non_blocking=True), pos.cuda(non_blocking=True), tab.cuda(non_blocking=True)
            nxt = self.llm.decode(ids_d, pos_d, tab_d, self.kv, max_ctx, stream=s)
            s.synchronize()
            now = time.perf_counter()
            out = nxt.cpu()
        for r, t in zip(batch, out.tolist()):
            r.last_token = t
            r.t_tokens.append(now)

    # ---------------------------------------------------------------- admission
    def _blocks_needed(self, req):
        return (self.n_vis + req.n_text + req.n_out + self.cfg.block - 1) // self.cfg.block

    def _prepare(self, req, ids_seed):
        need = self._blocks_needed(req)
        if need > self.max_blocks:
            raise nova.NovaError(nova.EINVAL, "request longer than the block table")
        if need > self.kv.num_blocks:
            raise nova.NovaError(nova.ENOKV, "request longer than the whole KV pool")
        req.ids = torch.from_numpy(synth.text_ids(req.n_text, self.cfg.vocab, seed=ids_seed)).to(self.device)

    def _reserve(self, req):
        """KV blocks for the whole request, taken when it is about to start vision encode; False
        (the request keeps waiting) while the pool has too few free blocks."""
        if req.blocks:
            return True
        need = self._blocks_needed(req)
        blocks = self.blocks.try_take(need)
        if blocks is None:
            return False
        req.blocks = blocks
        row = np.full(self.max_blocks, -1, np.int32)
        row[:need] = blocks
        req.table_row = row
        return True

    # ---------------------------------------------------------------- run
    def run(self, trace, seed=0):
        for r in trace:
            self._prepare(r, seed * 100003 + r.rid)
        if self.device == "cuda":
            torch.cuda.synchronize()
        if self.mode == "time_sliced":
            return self._run_sliced(trace)
        return self._run_threads(trace)

    def _run_threads(self, trace):
        vq, pq, dq = queue.Queue(), queue.Queue(), queue.Queue()
        stop = threading.Event()
        abort = threading.Event()

        def guarded(body):
            # a failed launch or a HIP error inside a worker must end the run, not leave the
            # scheduler waiting for an event that never comes
            def run():
                try:
                    body()
                except BaseException as exc:          # noqa: BLE001 -- re-raised by the scheduler
                    abort.set()
                    self.events.put(("error", exc))
            return run

        def vision_worker():
            while True:
                req = vq.get()
                if req is None:
                    return
                self._vision(req)
                self.events.put(("vision_done", req))

        def prefill_worker():
            while True:
                req = pq.get()
                if req is None:
                    return
                self._prefill(req)
                self.events.put(("prefill_done", req))

        def decode_worker():
            batch, waiting = [], []
            while not stop.is_set() or batch or waiting or not dq.empty():
                if abort.is_set():
                    return
                try:
                    while True:
                        waiting.append(dq.get(block=not batch and not waiting, timeout=0.01))
                except queue.Empty:
                    pass
                while waiting and len(batch) < self.max_batch:     # in-flight batching: join at a step boundary
                    batch.append(waiting.pop(0))
                if not batch:
                    continue
                self.decode_batches.append(len(batch))
                self._decode_step(batch)
                for r in [r for r in batch if r.done]:
                    batch.remove(r)
                    self.events.put(("finished", r))

        threads = [threading.Thread(target=guarded(f), daemon=True) for f in (vision_worker, prefill_worker, decode_worker)]
        for t in threads:
            t.start()
        t0 = time.perf_counter()
        pending_arrivals = list(trace)
        q_vision = []                 # Alg. 1 Q_v: vision requests waiting for encode/prefill to clear
        busy = {"vision": False, "prefill": False}
        finished = 0

        def try_vision():
            if q_vision and not busy["vision"] and not busy["prefill"] and self._reserve(q_vision[0]):
                r = q_vision.pop(0)
                busy["vision"] = True
                with self.lock:
                    self.other = nova.STAGE_ENCODE
                vq.put(r)

        while finished < len(trace):
            now = time.perf_counter() - t0
            while pending_arrivals and pending_arrivals[0].arrival <= now:
                r = pending_arrivals.pop(0)
                r.t_arrive = t0 + r.arrival
                with self.lock:
                    self.n_pending += 1
                q_vision.append(r)
                try_vision()
            timeout = max(0.0, pending_arrivals[0].arrival - now) if pending_arrivals else 0.05
            try:
                ev, r = self.events.get(timeout=min(timeout, 0.05))
            except queue.Empty:
                continue
            t_ev = time.perf_counter()
            if ev == "error":
                stop.set()
                vq.put(None)
                pq.put(None)
                for t in threads:
                    t.join(timeout=30)
                raise RuntimeError(f"serving worker failed: {r!r}") from r
            if ev == "vision_done":
                busy["vision"] = False
                busy["prefill"] = True            # prefill goes first, before any further vision
                with self.lock:
                    self.other = nova.STAGE_PREFILL
                pq.put(r)
            elif ev == "prefill_done":
                busy["prefill"] = False
                with self.lock:
                    self.n_pending -= 1
                    self.decode_active += 1
                    self.other = None
                r.t_tokens.append(r.t_pre1)      # prefill emits the first token
                if r.done:
                    self.events.put(("finished", r))
                else:
                    dq.put(r)
                try_vision()
            elif ev == "finished":
                with self.lock:
                    self.decode_active -= 1
                self.blocks.give(r.blocks)
                finished += 1
                try_vision()                      # freed KV blocks may admit the next request
            self.sched_us.append((time.perf_counter() - t_ev) * 1e6)
        stop.set()
        vq.put(None)
        pq.put(None)
        for t in threads:
            t.join(timeout=30)
        return self._summary(trace)

    def _slice_decode_next(self, n_batch, n_decode, other_ready, last_was_decode):
        """Whether the time-sliced driver runs a decode step next (rather than an encode/prefill pass).

        ``alternate``: a decode step between any two encode/prefill passes; ``decode_first``: decode
        whenever a batch is active; ``prefill_first``: encode/prefill whenever one is queued, decode
        otherwise, or (with ``decode_limit``, the paper's PF-Limit baseline) also once more than
        ``decode_limit`` requests are in the decode stage."""
        if n_batch == 0:
            return False
        if not other_ready:
            return True
        if self.slice_order == "decode_first":
            return True
        if self.slice_order == "prefill_first":
            return self.decode_limit is not None and n_decode > self.decode_limit
        return not last_was_decode

    def _run_sliced(self, trace):
        t0 = time.perf_counter()
        pending = list(trace)
        q_vision, q_prefill, q_decode, batch = [], [], [], []
        finished, last_was_decode = 0, False
        while finished < len(trace):
            now = time.perf_counter() - t0
            while pending and pending[0].arrival <= now:
                r = pending.pop(0)
                r.t_arrive = t0 + r.arrival
                q_vision.append(r)
            while q_decode and len(batch) < self.max_batch:   # join at a step boundary
                batch.append(q_decode.pop(0))
            vision_ready = bool(q_vision) and self.blocks.available() >= self._blocks_needed(q_vision[0])
            if self._slice_decode_next(len(batch), len(batch) + len(q_decode), bool(q_prefill) or vision_ready,
                                       last_was_decode):
                self.decode_batches.append(len(batch))
                self._decode_step(batch)
                last_was_decode = True
                for r in [r for r in batch if r.done]:
                    batch.remove(r)
                    self.blocks.give(r.blocks)
                    finished += 1
                continue
            last_was_decode = False
            if q_prefill:
                r = q_prefill.pop(0)
                self._prefill(r)
                r.t_tokens.append(r.t_pre1)
                if r.done:
                    self.blocks.give(r.blocks)
                    finished += 1
                else:
                    q_decode.append(r)
                continue
            if q_vision and self._reserve(q_vision[0]):
                r = q_vision.pop(0)
                self._vision(r)
                q_prefill.append(r)
                continue
            if pending:
                time.sleep(max(0.0, min(0.002, pending[0].arrival - (time.perf_counter() - t0))))
        return self._summary(trace)

    def _summary(self, trace):
        out = summarize(trace)
        bs = np.array(self.decode_batches or [0])
        out["decode_steps"] = int(len(self.decode_batches))
        out["avg_decode_batch"] = round(float(bs.mean()), 3)
        for key, vals in (("sched_event_us", self.sched_us), ("worker_partition_us", self.worker_us)):
            if vals:
                us = np.array(vals)
                out[key] = {f"p{q}": round(float(np.percentile(us, q)), 1) for q in (10, 50, 90, 99)}
                out[key].update(max=round(float(us.max()), 1), n=int(len(us)))
        return out


def summarize(trace, rate=None):
    """Latency and throughput of a finished trace.  The vision queue wait (arrival to the start of
    encode) is set beside Eq. 6's M/G/1 prediction from the measured service times T = encode +
    prefill (first moment and second moment) at the trace's arrival rate."""
    e2e = np.array([r.t_tokens[-1] - r.t_arrive for r in trace])
    ttft = np.array([r.t_pre1 - r.t_arrive for r in trace])
    tbt = np.array([np.mean(np.diff(r.t_tokens)) if len(r.t_tokens) > 1 else 0.0 for r in trace])
    qwait = np.array([r.t_vis0 - r.t_arrive for r in trace])
    service = np.array([r.t_pre1 - r.t_vis0 for r in trace])
    span = max(r.t_tokens[-1] for r in trace) - min(r.t_arrive for r in trace)
    lam = rate if rate is not None else len(trace) / max(trace[-1].arrival, 1e-9)
    pred = sched.mg1_wait(lam, float(service.mean()), float((service ** 2).mean()))
    return {"requests": len(trace), "max_e2e_s": round(float(e2e.max()), 4), "avg_e2e_s": round(float(e2e.mean()), 4),
            "p50_e2e_s": round(float(np.median(e2e)), 4), "avg_ttft_s": round(float(ttft.mean()), 4),
            "avg_tbt_ms": round(float(tbt.mean()) * 1e3, 3), "max_tbt_ms": round(float(tbt.max()) * 1e3, 3),
            "avg_queue_wait_s": round(float(qwait.mean()), 4), "throughput_req_s": round(len(trace) / span, 3),
            "mean_service_s": round(float(service.mean()), 4),
            "mean_service2_s2": round(float((service ** 2).mean()), 6),
            "eq6_predicted_wait_s": None if pred == float("inf") else round(pred, 4)}
