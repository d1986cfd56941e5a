"""Slot-level uplink emulation (test infrastructure only).

Communication model of Sec. III-A and the causal completion-event
generation of Sec. IV-B, written out slot by slot:

  * each agent k has a payload of B_k bits, Q_k[1] = B_k;
  * at the start of slot t the eligible set holds the agents with
    Q_k[t] > 0 and t >= l_k (eq. eligible_set);
  * every RB f is given to one eligible agent chosen by a causal policy
    (eqs. rb_orthogonality, pluggable_scheduler), or left idle;
  * agent k sends d_k[t] = Delta * sum_f x_{k,f}[t] R_{k,f}[t] bits
    (eq. slot_payload) and Q_k[t+1] = max(0, Q_k[t] - d_k[t])
    (eq. queue_evolution);
  * the slot in which Q_k first drops from positive to zero is the
    completion slot tau_k and a_k = tau_k * Delta (eqs. branch_arrival,
    completion_event); a branch still undelivered at the horizon leaves
    a_k = +inf and the frame is infeasible (Sec. IV-C).

Rates: R_{k,f}[t] = bandwidth * log2(1 + snr * g_{k,f}[t]) with
g ~ Exp(1) (Rayleigh fading power) drawn by ``synth.fading_draws`` (the
single-RB workloads), or the OFDMA channel of ``oracle.ofdma``.

Policies: round robin and proportional fair (single-RB workloads), and the
five causal evaluation schedulers of eqs. evaluation_schedulers and
evaluation_scores: RB f goes to the eligible agent with the largest score
s_{k,f}[t], ties to the smallest agent index, where s is
  MaxRate           R_{k,f}[t]
  MaxWeight         Q_k[t] R_{k,f}[t]
  EarliestRelease   -Q_k[t] / b_{k,f}[t],  b = Delta R_{k,f}[t] (the payload
                    RB f can deliver in slot t; -inf where it is 0)
  DAGRank           omega_k R_{k,f}[t]  (omega: normalised upward rank)
  TW-MaxRate        q_k R_{k,f}[t]      (q: fixed task weights)
Every RB of a slot is assigned from the slot-start state Q[t] (the causal
history of eq. causal_history holds Q[1:t], not the effect of the RBs of
the same slot), so one agent may receive several RBs of a slot.
"""

import math

import numpy as np
from scipy.special import exp1


def shannon_rates(gains, snr_db, bandwidth_hz):
    """[T, K, F] achievable rates in bit/s."""
    snr = 10.0 ** (snr_db / 10.0)
    return bandwidth_hz * np.log2(1.0 + snr * np.asarray(gains, dtype=np.float64))


def ergodic_rate(snr_db, bandwidth_hz):
    """E[bandwidth * log2(1 + snr X)], X ~ Exp(1):
    bandwidth * log2(e) * e^(1/snr) * E1(1/snr)."""
    snr = 10.0 ** (snr_db / 10.0)
    return bandwidth_hz * math.log2(math.e) * math.exp(1.0 / snr) * exp1(1.0 / snr)


class RoundRobin:
    """A pointer cycles over the agents in index order; each RB goes to the
    first eligible agent after the last one served.  The first RB of the
    first slot goes to the first eligible agent from index 0."""

    def __init__(self, K):
        self.last = -1
        self.K = K

    def pick(self, t, f, eligible, R, Q):
        for step in range(1, self.K + 1):
            k = (self.last + step) % self.K
            if k in eligible:
                self.last = k
                return k
        return None

    def end_slot(self, x, R):
        pass


class ProportionalFair:
    """k* = argmax R_k / Rbar_k over the eligible set, ties to the smallest
    index; after each slot every agent's average is updated as
    Rbar <- (1 - 1/W) Rbar + (1/W) * (rate it was served in the slot)."""

    def __init__(self, K, window, init_rate):
        self.W = float(window)
        self.avg = np.full(K, float(init_rate))

    def pick(self, t, f, eligible, R, Q):
        best, best_v = None, -np.inf
        for k in sorted(eligible):
            v = R[k, f] / self.avg[k]
            if v > best_v:
                best, best_v = k, v
        return best

    def end_slot(self, x, R):
        K, F = x.shape
        for k in range(K):
            served = 0.0
            for f in range(F):
                if x[k, f]:
                    served += R[k, f]
            self.avg[k] = (1.0 - 1.0 / self.W) * self.avg[k] + served / self.W


class ScoreArgmax:
    """Generic argmax policy over a per-agent score (eq.
    evaluation_schedulers); ties to the smallest index."""

    def __init__(self, score):
        self.score = score

    def pick(self, t, f, eligible, R, Q):
        best, best_v = None, None
        for k in sorted(eligible):
            v = self.score(k, f, R, Q)
            if best is None or v > best_v:
                best, best_v = k, v
        return best

    def end_slot(self, x, R):
        pass


def emulate(rates, B_bits, slot_s, policy, ell=None):
    """Run the slot loop.  ``rates`` is [T, K, F] bit/s, ``B_bits`` [K].

    Returns dict(a = arrival times in s (inf if undelivered), tau = completion
    slot (1-based, 0 if undelivered), d = [T, K] bits sent per slot,
    x = [T, K, F] allocation, feasible).
    """
    R = np.asarray(rates, dtype=np.float64)
    T, K, F = R.shape
    B = np.asarray(B_bits, dtype=np.float64)
    ell = np.ones(K, dtype=np.int64) if ell is None else np.asarray(ell)
    Q = B.copy()
    a = np.full(K, np.inf)
    tau = np.zeros(K, dtype=np.int64)
    d_all = np.zeros((T, K))
    x_all = np.zeros((T, K, F), dtype=np.int8)
    for ti in range(T):
        t = ti + 1
        eligible = {k for k in range(K) if Q[k] > 0 and t >= ell[k]}
        x = np.zeros((K, F), dtype=np.int8)
        if eligible:
            for f in range(F):
                k = policy.pick(t, f, eligible, R[ti], Q)
                x[k, f] = 1
        # eq. slot_payload: the rates of the RBs an agent holds, summed in
        # ascending RB order, times the slot length
        d = np.zeros(K)
        for k in range(K):
            acc = 0.0
            for f in range(F):
                if x[k, f]:
                    acc += R[ti, k, f]
            d[k] = slot_s * acc
        Qn = np.maximum(0.0, Q - d)
        for k in range(K):
            if Q[k] > 0 and Qn[k] == 0:
                tau[k] = t
                a[k] = t * slot_s
        policy.end_slot(x, R[ti])
        d_all[ti] = d
        x_all[ti] = x
        Q = Qn
        if np.all(np.isfinite(a)):
            d_all = d_all[:t]
            x_all = x_all[:t]
            break
    return dict(a=a, tau=tau, d=d_all, x=x_all, feasible=bool(np.all(np.isfinite(a))))


def _earliest_release(slot_s):
    def score(k, f, R, Q):
        b = slot_s * R[k, f]
        return -Q[k] / b if b > 0.0 else -math.inf
    return score


def make_policy(name, K, snr_db=None, bandwidth_hz=None, window=100, slot_s=None, weights=None):
    """Policy by name: rr, pf, maxrate, maxweight, earliest_release (needs
    slot_s), dagrank and tw_maxrate (need the per-agent weights)."""
    if name == "rr":
        return RoundRobin(K)
    if name == "pf":
        return ProportionalFair(K, window, ergodic_rate(snr_db, bandwidth_hz))
    if name == "maxrate":
        return ScoreArgmax(lambda k, f, R, Q: R[k, f])
    if name == "maxweight":
        return ScoreArgmax(lambda k, f, R, Q: Q[k] * R[k, f])
    if name == "earliest_release":
        return ScoreArgmax(_earliest_release(float(slot_s)))
    if name in ("dagrank", "tw_maxrate"):
        w = [float(v) for v in weights]
        return ScoreArgmax(lambda k, f, R, Q: w[k] * R[k, f])
    raise ValueError(name)


def trace_arrivals(cfg, gains, B_bytes, snr_db, scheduler):
    """Arrival vector (s) of one uplink trace of a config."""
    arr = cfg["arrivals"]
    R = shannon_rates(gains, snr_db, arr["bandwidth_hz"])
    pol = make_policy(scheduler, cfg["K"], snr_db, arr["bandwidth_hz"], arr["pf_window"])
    return emulate(R, np.asarray(B_bytes, dtype=np.float64) * 8.0, arr["slot_s"], pol)
