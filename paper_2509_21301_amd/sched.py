"""Partition planning for co-running stages (the paper's Sec. 3.3): expected end-to-end latency
of an ideal pipeline (Eq. 1-2), the enumeration of the best static partition (Eq. 3), the
throughput approximation (Eq. 4), the latency-throughput Pareto front, the adaptive decode
share (Eq. 5), and the choice of a Pareto point for a request rate using the M/G/1 queueing
delay of the encode + prefill server (Eq. 6), all driven by measured per-stage curves.

A partition here is the number of CUs the decode stage holds while it co-runs with vision
encode (P_v) or with prefill (P_p); the co-running stage holds the rest of the 256.  On
gfx950 a partition is a whole number of XCD-balanced mask groups (8 CUs = one per XCD).
"""
from __future__ import annotations

from dataclasses import dataclass, field

TOTAL_CUS = 256
GRANULE = 8


@dataclass
class StageCurves:
    """Measured co-run times (seconds) indexed by the decode CU count."""
    shares: list[int]
    t_vision: dict[int, float]          # encode pass while decode holds the share
    t_prefill: dict[int, float]         # prefill pass while decode holds the share
    t_dec_vision: dict[int, float]      # decode step while co-running with encode
    t_dec_prefill: dict[int, float]     # decode step while co-running with prefill

    @classmethod
    def from_corun(cls, records):
        """Build from bench.py's `corun` records (milliseconds)."""
        tv, tp, dv, dp, shares = {}, {}, {}, {}, set()
        for r in records:
            p = r["decode_cus"]
            shares.add(p)
            if r["pair"] == "decode+encode":
                tv[p] = r["encode_ms_corun"] / 1e3
                dv[p] = r["decode_step_ms_corun"] / 1e3
            else:
                tp[p] = r["prefill_ms_corun"] / 1e3
                dp[p] = r["decode_step_ms_corun"] / 1e3
        return cls(sorted(shares), tv, tp, dv, dp)


def expected_e2e(c: StageCurves, pv: int, pp: int, out_len: float) -> float:
    """Eq. 1 with the co-run proportions of Eq. 2."""
    tv, tp = c.t_vision[pv], c.t_prefill[pp]
    share_v = tv / (tv + tp)
    return tv + tp + (share_v * c.t_dec_vision[pv] + (1.0 - share_v) * c.t_dec_prefill[pp]) * out_len


def ideal_throughput(c: StageCurves, pv: int, pp: int) -> float:
    """Eq. 4: requests per second when encode and prefill run back to back."""
    return 1.0 / (c.t_vision[pv] + c.t_prefill[pp])


def best_static(c: StageCurves, out_len: float):
    """Eq. 3: (P_v, P_p, latency) minimising Eq. 1 over all measured partition pairs."""
    best = None
    for pv in c.shares:
        for pp in c.shares:
            lat = expected_e2e(c, pv, pp, out_len)
            if best is None or lat < best[2]:
                best = (pv, pp, lat)
    return best


def pareto_front(c: StageCurves, out_len: float):
    """Partition pairs whose (latency, throughput) no other pair improves on both counts.
    Returns [(latency, throughput, P_v, P_p)] sorted by latency."""
    pts = [(expected_e2e(c, a, b, out_len), ideal_throughput(c, a, b), a, b) for a in c.shares for b in c.shares]
    pts.sort(key=lambda t: (t[0], -t[1]))
    front, best_thr = [], -1.0
    for p in pts:
        if p[1] > best_thr:
            front.append(p)
            best_thr = p[1]
    return front


def queue_wait(t_service: float, rate: float) -> float:
    """Eq. 6 for a service time that is the same for every request (E[T^2] = T^2): the expected
    wait in the vision queue at `rate` requests/s; infinite when the server is saturated."""
    rho = rate * t_service
    return float("inf") if rho >= 1.0 else rate * t_service * t_service / (2.0 * (1.0 - rho))


def mg1_wait(rate: float, mean_t: float, mean_t2: float) -> float:
    """Eq. 6 with measured moments of the service time T = t_vision + t_prefill:
    lambda E[T^2] / (2 (1 - lambda E[T])); infinite when the server is saturated."""
    rho = rate * mean_t
    return float("inf") if rho >= 1.0 else rate * mean_t2 / (2.0 * (1.0 - rho))


def best_under_load(c: StageCurves, out_len: float, rate: float):
    """The partition pair minimising Eq. 1 plus the Eq. 6 queueing delay at `rate` (the Pareto
    point the request rate calls for: fewer decode CUs as the rate grows).  Returns
    (P_v, P_p, latency); when every pair saturates, the pair of highest throughput (Eq. 4)."""
    best = None
    for pv in c.shares:
        for pp in c.shares:
            lat = expected_e2e(c, pv, pp, out_len) + queue_wait(c.t_vision[pv] + c.t_prefill[pp], rate)
            if best is None or lat < best[2]:
                best = (pv, pp, lat)
    if best[2] == float("inf"):
        pv, pp = max(((a, b) for a in c.shares for b in c.shares), key=lambda ab: ideal_throughput(c, *ab))
        best = (pv, pp, float("inf"))
    return best


def decode_cus(n_pending: int, optimum: int, alpha: int, minimum: int, granule: int = GRANULE) -> int:
    """Eq. 5: decode's CUs shrink by alpha per pending encode/prefill request beyond the first,
    never below the floor; rounded down to the mask granule."""
    cus = max(minimum, optimum - alpha * (max(n_pending, 1) - 1))
    return max(granule, cus // granule * granule)


def on_granule(c: StageCurves, granule: int = GRANULE) -> StageCurves:
    """The curves at every multiple of `granule` between the smallest and largest measured
    shares, linear between measured neighbours (masks come in steps of one CU per XCD)."""
    pts = sorted(c.shares)
    grid = list(range(pts[0], pts[-1] + 1, granule))

    def lerp(d):
        out = {}
        for p in grid:
            hi = next(q for q in pts if q >= p)
            lo = max(q for q in pts if q <= p)
            out[p] = d[lo] if hi == lo else d[lo] + (d[hi] - d[lo]) * (p - lo) / (hi - lo)
        return out
    return StageCurves(grid, lerp(c.t_vision), lerp(c.t_prefill), lerp(c.t_dec_vision), lerp(c.t_dec_prefill))


def adaptive_params(c: StageCurves, out_len: float, rates, granule: int = GRANULE, tbt_factor: float = 2.0):
    """Hyperparameters of Eq. 5 from the measured curves (Sec. 3.3.2; the paper picks them per
    stage pair from its Pareto analysis, Sec. 5.1):

    * SM_op: Eq. 3's optimum for each pair (decode beside encode, decode beside prefill);
    * for each rate, the Pareto point it calls for (Eq. 1 plus the Eq. 6 wait, best_under_load)
      gives a decode share, and Little's law gives the requests pending in encode / prefill,
      N = rate * (E[W_q] + E[T]);
    * alpha: the least-squares slope of SM_op - share against N - 1 over the rates with N > 1
      (Eq. 5's linear decrease), rounded to whole CUs, never negative;
    * SM_min: the smallest share whose co-run decode step stays within tbt_factor times the step
      at SM_op (the floor bounds TBT).
    All on the granule-interpolated curves.  Returns a dict, with the per-rate points."""
    g = on_granule(c, granule)
    op_v, op_p, _ = best_static(g, out_len)
    pts = []
    for r in rates:
        pv, pp, lat = best_under_load(g, out_len, r)
        t = g.t_vision[pv] + g.t_prefill[pp]
        w = queue_wait(t, r)
        if w == float("inf"):
            continue
        pts.append({"rate": r, "decode_cus_with_encode": pv, "decode_cus_with_prefill": pp,
                    "pending": r * (w + t), "expected_e2e_s": lat})

    def slope(op, key):
        num = sum((op - q[key]) * (q["pending"] - 1) for q in pts if q["pending"] > 1)
        den = sum((q["pending"] - 1) ** 2 for q in pts if q["pending"] > 1)
        return max(0, int(round(num / den))) if den > 0 else 0

    def floor(op, dec):
        lim = tbt_factor * dec[op]
        return min(p for p in g.shares if dec[p] <= lim)
    return {"sm_op_v": op_v, "sm_op_p": op_p,
            "alpha_v": slope(op_v, "decode_cus_with_encode"), "alpha_p": slope(op_p, "decode_cus_with_prefill"),
            "sm_min": max(floor(op_v, g.t_dec_vision), floor(op_p, g.t_dec_prefill), granule),
            "granule": granule, "tbt_factor": tbt_factor, "points": pts}
