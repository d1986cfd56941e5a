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

The slot loop itself runs in the library (rtcc_uplink_emulate): round
robin, proportional fair (average initialised at the ergodic rate of the
Rayleigh channel), and the five causal evaluation schedulers (MaxRate,
MaxWeight, EarliestRelease, DAGRank, Task-Weighted MaxRate; eqs.
evaluation_schedulers, evaluation_scores).  This module computes the rates
and the ergodic-rate closed form.
"""

import math

import numpy as np

from . import rtcc as R


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


SCHEDULERS = {
    "rr": R.RTCC_SCHED_ROUND_ROBIN,
    "pf": R.RTCC_SCHED_PROPORTIONAL_FAIR,
    "maxrate": R.RTCC_SCHED_MAXRATE,
    "maxweight": R.RTCC_SCHED_MAXWEIGHT,
    "earliest_release": R.RTCC_SCHED_EARLIEST_RELEASE,
    "dagrank": R.RTCC_SCHED_WEIGHTED_RATE,
    "tw_maxrate": R.RTCC_SCHED_WEIGHTED_RATE,
}


def completion_slots(rates, payload_bits, slot_s, scheduler, agent_weight=None, pf_window=100.0,
                     pf_init_rate=1.0, kind="gpu"):
    """Completion slot per agent (0 = undelivered) of the native slot-level
    emulation (rtcc_uplink_emulate) for a [slots, K, RBs] rate array."""
    return R.rtcc_uplink_emulate(rates, payload_bits, SCHEDULERS[scheduler], slot_s, agent_weight=agent_weight,
                                 pf_window=pf_window, pf_init_rate=pf_init_rate, kind=kind)


def completion_times(gains, payload_bits, snr_db, bandwidth_hz, slot_s, scheduler, pf_window=100, kind="gpu"):
    """Arrival time per agent (s), inf if undelivered within the slots of
    ``gains`` ([slots, K, RBs] power gains), for the Shannon-rate channel."""
    g = np.asarray(gains, dtype=np.float64)
    rate = bandwidth_hz * np.log2(1.0 + (10.0 ** (snr_db / 10.0)) * g)
    slots = completion_slots(rate, payload_bits, slot_s, scheduler, pf_window=float(pf_window),
                             pf_init_rate=mean_rate(snr_db, bandwidth_hz), kind=kind)
    return np.where(slots > 0, slots * slot_s, np.inf)
