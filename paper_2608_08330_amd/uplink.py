"""Slot-level uplink emulation that produces branch completion times.

Communication model of Sec. III-A with causal completion events (Sec.
IV-B): per slot the eligible agents are those with undelivered payload
(eq. eligible_set, local availability at slot 1); each resource block goes
to one eligible agent chosen by a causal policy (eq. pluggable_scheduler);
an agent on a block sends rate * slot bits (eq. slot_payload); its backlog
drops by that amount, floored at zero (eq. queue_evolution); the slot in
which the backlog reaches zero is the completion slot, and a_k = slot *
slot duration (eqs. branch_arrival, completion_event).  Undelivered at the
horizon -> infeasible frame.

Policies: round robin over the eligible agents (next after the last served)
and proportional fair (argmax of instantaneous rate over an exponentially
weighted average rate with window W, ties to the smallest index, average
initialised at the ergodic rate of the Rayleigh channel).
"""

import math

import numpy as np


def _expint_e1(x):
    """Exponential integral E1(x), x > 0: power series for x <= 1, Lentz
    continued fraction otherwise (Abramowitz & Stegun 5.1.11, 5.1.22)."""
    if x <= 1.0:
        s, term, k = 0.0, 1.0, 1
        while True:
            term *= -x / k
            add = -term / k
            s += add
            if abs(add) < 1e-17 * abs(s) + 1e-300:
                break
            k += 1
        return -0.5772156649015329 - math.log(x) + s
    b = x + 1.0
    c = 1.0 / 1e-300
    d = 1.0 / b
    h = d
    i = 1
    while True:
        an = -i * i
        b += 2.0
        d = 1.0 / (an * d + b)
        c = b + an / c
        de = c * d
        h *= de
        if abs(de - 1.0) < 1e-16:
            break
        i += 1
    return h * math.exp(-x)


def mean_rate(snr_db, bandwidth_hz):
    """Ergodic Shannon rate of a Rayleigh channel, bit/s:
    B log2(e) e^(1/snr) E1(1/snr)."""
    snr = 10.0 ** (snr_db / 10.0)
    return bandwidth_hz * math.log2(math.e) * math.exp(1.0 / snr) * _expint_e1(1.0 / snr)


def completion_times(gains, payload_bits, snr_db, bandwidth_hz, slot_s, scheduler, pf_window=100):
    """Arrival time per agent (s), inf if undelivered within the slots of
    ``gains`` ([slots, K, RBs] power gains)."""
    g = np.asarray(gains, dtype=np.float64)
    T, K, F = g.shape
    rate = bandwidth_hz * np.log2(1.0 + (10.0 ** (snr_db / 10.0)) * g)
    backlog = np.asarray(payload_bits, dtype=np.float64).copy()
    arrival = np.full(K, np.inf)
    last = -1
    avg = np.full(K, mean_rate(snr_db, bandwidth_hz))
    for t in range(T):
        active = backlog > 0
        if not active.any():
            break
        served_rate = np.zeros(K)
        for f in range(F):
            if scheduler == "rr":
                k = -1
                for step in range(1, K + 1):
                    c = (last + step) % K
                    if active[c]:
                        k = c
                        break
                last = k
            elif scheduler == "pf":
                score = np.where(active, rate[t, :, f] / avg, -np.inf)
                k = int(np.argmax(score))
            else:
                raise ValueError(scheduler)
            served_rate[k] += rate[t, k, f]
        sent = served_rate * slot_s
        new = np.maximum(0.0, backlog - sent)
        done = active & (new == 0.0)
        arrival[done] = (t + 1) * slot_s
        backlog = new
        if scheduler == "pf":
            avg = (1.0 - 1.0 / pf_window) * avg + served_rate / pf_window
    return arrival
