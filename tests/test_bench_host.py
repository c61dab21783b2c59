"""bench.py's serving harness on the host, with the GPU passes replaced by timed stand-ins (the
fake server of test_serve_policy): every mode runs on the same traces, the summary pools the
seeds per (mode, rate), picks the better time-sliced order, and sets Eq. 6 beside the wait."""
import numpy as np

import bench
from paper_2509_21301_amd import sched, serve
from tests.test_sched_host import curves
from tests.test_serve_policy import fake_server


class FakeSetup:
    """ServingSetup's serve() over the fake server."""

    def serve(self, kw, trace, keep_log=False):
        kw = dict(kw)
        srv, _ = fake_server(kw.pop("mode"), **{k: kw.pop(k) for k in ("slice_order", "decode_limit") if k in kw})
        srv.decode_cus = kw.get("decode_cus", srv.decode_cus)
        srv.alpha = kw.get("alpha", srv.alpha)
        srv.minimum = kw.get("minimum", srv.minimum)
        res = srv.run(trace)
        if keep_log:
            res["partition_timeline"] = [[round(t * 1e3, 2), st, cus] for t, st, cus in srv.partition_log]
            res["arrivals_ms"] = [r.arrival * 1e3 for r in trace]
        return res


def test_run_serving_summary(monkeypatch):
    small = serve.poisson_trace
    monkeypatch.setattr(serve, "poisson_trace", lambda rate, window, seed: small(rate, window, seed, n_text=(5, 9),
                                                                                   n_out=(6, 12)))
    monkeypatch.setattr(serve.nova, "make_cu_mask", lambda n, first=0: [0xFFFFFFFF] * 8)
    monkeypatch.setattr(serve.nova, "set_stage_partition", lambda stage, mask: None)
    out = bench.run_serving(serve, sched, FakeSetup(), curves(2), 32, [100.0], [1, 2], 0.05, timeline_at=(100.0, 1))
    modes = {r["mode"] for r in out["runs"]}
    assert modes == {"nova_rate_static", "nova_adaptive", "time_sliced_decode_first", "time_sliced_prefill_first",
                     "pf_limit", "multi_stream"}
    assert len(out["runs"]) == 12
    rows = {r["mode"]: r for r in out["summary"]}
    best = rows["time_sliced_best"]
    assert best["chosen"] in ("time_sliced_decode_first", "time_sliced_prefill_first")
    assert best["max_e2e_s"] == min(rows["time_sliced_decode_first"]["max_e2e_s"],
                                    rows["time_sliced_prefill_first"]["max_e2e_s"])
    for m in modes:
        rs = [r for r in out["runs"] if r["mode"] == m]
        assert abs(rows[m]["max_e2e_s"] - np.mean([r["max_e2e_s"] for r in rs])) < 1e-3
        assert rows[m]["seeds"] == 2 and "eq6_predicted_wait_s" in rows[m]
    assert any("partition_timeline" in r for r in out["runs"] if r["mode"] == "nova_adaptive")
    a = out["adaptive_params"]
    assert a["sm_min"] <= min(a["sm_op_v"], a["sm_op_p"])
