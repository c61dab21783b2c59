"""Host-side partition planning (paper_2509_21301_amd.sched) against the oracle's statement of
Eq. 1-5 on the same curves (the two are written independently)."""
import numpy as np

from oracle import sched as osched
from paper_2509_21301_amd import sched

SHARES = [32, 64, 96, 128, 160, 192, 224]


def curves(seed):
    r = np.random.default_rng(seed)
    tv = {p: 0.03 * 256 / (256 - p) * (1 + 0.1 * r.random()) for p in SHARES}
    tp = {p: 0.02 * 256 / (256 - p) * (1 + 0.1 * r.random()) for p in SHARES}
    dv = {p: 0.004 * 256 / p * (1 + 0.2 * r.random()) for p in SHARES}
    dp = {p: 0.005 * 256 / p * (1 + 0.2 * r.random()) for p in SHARES}
    return sched.StageCurves(SHARES, tv, tp, dv, dp)


def test_e2e_and_best_static_match_oracle():
    for seed in range(5):
        c = curves(seed)
        for out_len in (16, 32, 48):
            for pv in SHARES:
                for pp in SHARES:
                    ref = osched.e2e_latency(c.t_vision[pv], c.t_prefill[pp], c.t_dec_vision[pv], c.t_dec_prefill[pp], out_len)
                    assert abs(sched.expected_e2e(c, pv, pp, out_len) - ref) < 1e-12
            pv, pp, lat = sched.best_static(c, out_len)
            opv, opp, olat = osched.optimal_partition(SHARES, c.t_vision, c.t_prefill, c.t_dec_vision,
                                                      c.t_dec_prefill, out_len)
            assert (pv, pp) == (opv, opp) and abs(lat - olat) < 1e-12


def test_pareto_front_matches_oracle():
    c = curves(11)
    front = sched.pareto_front(c, 32)
    pts = [(sched.expected_e2e(c, a, b, 32), sched.ideal_throughput(c, a, b), (a, b)) for a in SHARES for b in SHARES]
    ref = osched.pareto_front(pts)
    assert [(f[2], f[3]) for f in front] == [p[2] for p in ref]
    lats = [f[0] for f in front]
    thrs = [f[1] for f in front]
    assert lats == sorted(lats) and thrs == sorted(thrs)
    assert abs(front[0][1] - osched.throughput(c.t_vision[front[0][2]], c.t_prefill[front[0][3]])) < 1e-12


def test_decode_share_eq5():
    for n in range(1, 8):
        assert sched.decode_cus(n, 96, 16, 32) == osched.decode_share(96, 16, 32, n)
    assert sched.decode_cus(0, 96, 16, 32) == 96
    assert sched.decode_cus(2, 100, 4, 12) == 96           # rounded down to the 8-CU granule
    assert sched.decode_cus(9, 100, 40, 4) == 8


def test_from_corun_records():
    recs = [{"pair": "decode+encode", "decode_cus": 64, "encode_ms_corun": 50.0, "decode_step_ms_corun": 12.0},
            {"pair": "decode+prefill", "decode_cus": 64, "prefill_ms_corun": 56.0, "decode_step_ms_corun": 12.5}]
    c = sched.StageCurves.from_corun(recs)
    assert c.shares == [64] and c.t_vision[64] == 0.05 and c.t_dec_prefill[64] == 0.0125


def test_best_under_load_matches_eq1_plus_eq6():
    c = curves(3)
    for rate in (0.5, 2.0, 5.0):
        pv, pp, lat = sched.best_under_load(c, 32, rate)
        ref = []
        for a in SHARES:
            for b in SHARES:
                t = c.t_vision[a] + c.t_prefill[b]
                w = osched.mg1_wait(rate, t, t * t) if rate * t < 1 else float("inf")
                ref.append((osched.e2e_latency(c.t_vision[a], c.t_prefill[b], c.t_dec_vision[a], c.t_dec_prefill[b], 32) + w, a, b))
        r = min(ref)
        assert (pv, pp) == (r[1], r[2]) and abs(lat - r[0]) < 1e-12
    # a higher rate never hands decode more CUs in total
    lo, hi = sched.best_under_load(c, 32, 0.1), sched.best_under_load(c, 32, 6.0)
    assert hi[0] + hi[1] <= lo[0] + lo[1]
    assert sched.queue_wait(0.2, 5.0) == float("inf")


def test_mg1_wait_matches_oracle():
    # Eq. 6 with measured first and second moments of the service time, and the saturated case
    for lam, t, t2 in [(2.0, 0.1, 0.012), (4.0, 0.2, 0.05), (0.5, 1.0, 1.5), (3.9, 0.25, 0.07)]:
        want = osched.mg1_wait(lam, t, t2)
        assert abs(sched.mg1_wait(lam, t, t2) - want) <= 1e-12 * max(1.0, abs(want))
    assert sched.mg1_wait(4.0, 0.25, 0.1) == float("inf")
    # deterministic service reduces to the fixed-T form used by the rate-aware search
    assert abs(sched.mg1_wait(3.0, 0.2, 0.04) - sched.queue_wait(0.2, 3.0)) < 1e-12


def test_curves_on_the_8_cu_granule():
    c = curves(4)
    g = sched.on_granule(c)
    assert g.shares == list(range(32, 225, 8))
    for p in SHARES:                                          # measured points kept exactly
        assert g.t_vision[p] == c.t_vision[p] and g.t_dec_prefill[p] == c.t_dec_prefill[p]
    assert abs(g.t_vision[40] - (0.75 * c.t_vision[32] + 0.25 * c.t_vision[64])) < 1e-15
    assert abs(g.t_dec_vision[112] - 0.5 * (c.t_dec_vision[96] + c.t_dec_vision[128])) < 1e-15


def test_adaptive_params_from_the_pareto_points():
    """Eq. 5's SM_op, alpha and SM_min derived from the curves: SM_op is Eq. 3's optimum on the
    granule curves, the rate-aware decode shares never grow with the rate, alpha is the
    least-squares slope of their decrease against the pending count, and the floor keeps the
    decode step within the TBT bound."""
    c = curves(7)
    rates = [0.5, 1, 2, 4, 6, 8, 10]
    a = sched.adaptive_params(c, 32, rates)
    g = sched.on_granule(c)
    pv, pp, _ = sched.best_static(g, 32)
    assert (a["sm_op_v"], a["sm_op_p"]) == (pv, pp)
    pts = a["points"]
    assert len(pts) >= 3 and all(q["pending"] > 0 for q in pts)
    shares = [q["decode_cus_with_encode"] + q["decode_cus_with_prefill"] for q in pts]
    assert shares == sorted(shares, reverse=True)
    for key, op, alpha in (("decode_cus_with_encode", pv, a["alpha_v"]), ("decode_cus_with_prefill", pp, a["alpha_p"])):
        xs = np.array([q["pending"] - 1 for q in pts if q["pending"] > 1])
        ys = np.array([op - q[key] for q in pts if q["pending"] > 1])
        want = max(0, int(round((xs * ys).sum() / (xs * xs).sum()))) if len(xs) else 0
        assert alpha == want
    assert 8 <= a["sm_min"] <= min(pv, pp)
    assert g.t_dec_vision[a["sm_min"]] <= 2.0 * g.t_dec_vision[pv] or g.t_dec_prefill[a["sm_min"]] <= 2.0 * g.t_dec_prefill[pp]
    # Little's law for one point by hand
    q = pts[0]
    t = g.t_vision[q["decode_cus_with_encode"]] + g.t_prefill[q["decode_cus_with_prefill"]]
    assert abs(q["pending"] - q["rate"] * (osched.mg1_wait(q["rate"], t, t * t) + t)) < 1e-9
