"""Oracle for the partition and scheduling formulas of the method (TEST INFRASTRUCTURE ONLY).

Each function writes out one formula of Sec. 3.3-3.5 as stated there; the HIP path's host
logic implements the same formulas independently.
"""
from __future__ import annotations

import itertools


def prop_weights(t_v, t_p):
    """Eq. 2: shares of the decode iterations that co-run with vision encode and with prefill."""
    return t_v / (t_v + t_p), t_p / (t_v + t_p)


def e2e_latency(t_v, t_p, t_d_v, t_d_p, out_len):
    """Eq. 1: ideal-pipeline expected end-to-end latency.

    t_v, t_p: vision-encode and prefill forward times under their partitions;
    t_d_v, t_d_p: decode iteration times while co-running with vision / prefill;
    out_len: number of generated tokens L.
    """
    pv, pp = prop_weights(t_v, t_p)
    return t_v + t_p + (pv * t_d_v + pp * t_d_p) * out_len


def throughput(t_v, t_p):
    """Eq. 4: request throughput when encode and prefill run back to back and decode overlaps them."""
    return 1.0 / (t_v + t_p)


def optimal_partition(shares, t_v, t_p, t_d_v, t_d_p, out_len):
    """Eq. 3: enumerate (P_v, P_p) over the valid partitions, minimising Eq. 1.

    ``shares`` is the list of valid partitions; t_v, t_p, t_d_v, t_d_p map a partition to the
    profiled times (t_d_v[P] is decode's time when vision holds P).  Returns (P_v, P_p, latency).
    """
    best = None
    for pv, pp in itertools.product(shares, shares):
        lat = e2e_latency(t_v[pv], t_p[pp], t_d_v[pv], t_d_p[pp], out_len)
        if best is None or lat < best[2]:
            best = (pv, pp, lat)
    return best


def pareto_front(points):
    """Latency-throughput Pareto front (Sec. 3.3.2): points (latency, throughput, tag) that no
    other point beats on both lower latency and higher throughput (with one strictly better)."""
    front = []
    for a in points:
        dominated = any((b[0] <= a[0] and b[1] >= a[1]) and (b[0] < a[0] or b[1] > a[1]) for b in points)
        if not dominated:
            front.append(a)
    return sorted(front, key=lambda p: p[0])


def decode_share(sm_op, alpha, sm_min, n_pend):
    """Eq. 5: decode's compute units given N_pend requests in vision encode or prefill."""
    return max(sm_min, sm_op - alpha * (n_pend - 1))


def mg1_wait(lam, mean_t, mean_t2):
    """Eq. 6: M/G/1 expected queueing delay, lambda E[T^2] / (2 (1 - lambda E[T]))."""
    return lam * mean_t2 / (2.0 * (1.0 - lam * mean_t))


def next_layer(cur, k, n_layers):
    """Eq. 7: the logical layer swapped into a physical slot after ``cur`` finishes."""
    return (cur + k) % n_layers


def ring_slots(n_layers, k, passes):
    """Sec. 3.5 stepped pass by pass: physical slots start with logical layers 0..K-1; when a
    layer's forward finishes, its slot takes the Eq. 7 successor.  Returns the layer each slot
    holds after ``passes`` full forward passes."""
    slots = list(range(k))
    for _ in range(passes):
        for layer in range(n_layers):
            slot = slots.index(layer)
            slots[slot] = next_layer(layer, k, n_layers)
    return slots


def offload_ok(size, t_fwd, bandwidth, n_layers, k):
    """Eq. 8 stated per layer: for every l in [K+1, L] the copy of (l-K)/L of the weights
    (size S at bandwidth B) must fit in the (l-2)/L of the forward time T before layer l."""
    return all((l - 2) / n_layers * t_fwd >= size / bandwidth * (l - k) / n_layers
               for l in range(k + 1, n_layers + 1))


def offload_min_bandwidth(size, t_fwd, n_layers, k):
    """The bound Eq. 8 yields: B >= S/T * (L - K)/(L - 2)."""
    return size / t_fwd * (n_layers - k) / (n_layers - 2)
