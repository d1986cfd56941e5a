"""OFDMA uplink channel of the evaluation and the measured-DAG trial
(test infrastructure only; see ``oracle/__init__.py``).

Channel (Sec. V-A2).  K agents move inside a W x H area whose centre hosts
the edge server; slot t (1-based) lasts Delta.  The rate of agent k on RB f
in slot t is its reference rate scaled by the channel effects the paper
lists (distance-dependent attenuation with exponent alpha, agent-specific
blockage, slot-level and RB-dependent small-scale variation) and by the
bandwidth factor beta:

  R_{k,f}[t] = beta * Rref_{k,f} * G(d_k[t]) * Z_k[t] * h_{k,f}[t]

Readings where the paper gives only the names of the effects:
  * rates scale linearly with the channel power gain (the low-SNR regime of
    the Shannon rate), so every effect is a power factor multiplying the
    reference rate, applied in the order written above;
  * position at the start of slot t: p_k + v_k (t - 1) Delta, straight
    motion at constant speed reflected at the area boundary;
  * G(d) = min(1, (d_ref / d)^alpha): the reference rate holds within the
    reference distance d_ref of the server;
  * blockage: a two-state chain per agent, blocked in slot 1 iff
    u0_k < rho (rho = long-run blocked fraction); from slot t-1 to slot t a
    blocked agent clears iff u_k[t] < 1 / D (D = mean blocked dwell in
    slots) and a clear agent becomes blocked iff u_k[t] < rho / ((1 - rho) D)
    (so that rho is the stationary fraction); a blocked agent's power is
    reduced by L_b dB, Z = 10^(-L_b / 10), else Z = 1;
  * h_{k,f}[t] ~ Exp(1) i.i.d. over agents, RBs and slots (Rayleigh block
    fading, independent across RBs: frequency selective).
Payload: B_k = gamma * (bytes of agent k's branch input) * 8 bits.

Measured-DAG trial (Sec. V-C): one channel trace, one (gamma, beta) and one
scheduler give the arrival vector a (eq. branch_arrival, through
``oracle.uplink.emulate``); RTCC (r = a) and Barrier (r = A) run on the
single-stream model with the profiled service times (``oracle.schedule``);
the gain T_B - T_R equals the pre-arrival encoder work W_pre.  Times are
integer nanoseconds, so the identity is checked exactly.  DAGRank weights
omega are the upward ranks (longest path to the exit, node costs included)
of the encoders in the profiled DAG, normalised by their maximum.
"""

import math

import numpy as np

from . import schedule as S
from . import uplink as U


def reflect(x, length):
    """Mirror-fold a coordinate into [0, length] (reflection at both walls)."""
    u = x % (2.0 * length)
    return u if u <= length else 2.0 * length - u


def position(draw, arr, k, t):
    """Position (m) of agent k at the start of slot t (1-based)."""
    tau = (t - 1) * arr["slot_s"]
    v, h = float(draw["speed_mps"][k]), float(draw["heading"][k])
    x = float(draw["pos0_m"][k, 0]) + v * math.cos(h) * tau
    y = float(draw["pos0_m"][k, 1]) + v * math.sin(h) * tau
    return reflect(x, arr["area_m"][0]), reflect(y, arr["area_m"][1])


def path_gain(d, arr):
    """min(1, (d_ref / d)^alpha); 1 at d = 0."""
    d_ref = arr["ref_distance_m"]
    if d <= d_ref:
        return 1.0
    return (d_ref / d) ** arr["path_loss_exp"]


def blockage(draw, arr, T, K):
    """[T][K] booleans: agent k blocked in slot t+1 (0-based row t)."""
    rho, D = arr["blockage_fraction"], arr["blockage_dwell_slots"]
    p_clear = 1.0 / D
    p_block = rho / ((1.0 - rho) * D)
    st = [[False] * K for _ in range(T)]
    for k in range(K):
        st[0][k] = bool(draw["block_u0"][k] < rho)
        for t in range(1, T):
            u = draw["block_u"][t, k]
            st[t][k] = (not (u < p_clear)) if st[t - 1][k] else bool(u < p_block)
    return st


def rates(draw, cfg, beta):
    """[T, K, F] rates in bit/s of one channel trace at bandwidth scale beta."""
    arr = cfg["arrivals"]
    T, K, F = arr["t_max_slots"], cfg["K"], arr["n_rb"]
    blocked = blockage(draw, arr, T, K)
    zb = 10.0 ** (-arr["blockage_loss_db"] / 10.0)
    sx, sy = arr["server_m"]
    R = np.zeros((T, K, F))
    for t in range(1, T + 1):
        for k in range(K):
            x, y = position(draw, arr, k, t)
            g = path_gain(math.hypot(x - sx, y - sy), arr)
            z = zb if blocked[t - 1][k] else 1.0
            for f in range(F):
                R[t - 1, k, f] = beta * float(draw["ref_rate_bps"][k, f]) * g * z * float(draw["fading"][t - 1, k, f])
    return R


def payload_bits(cfg, points_per_agent, gamma):
    """B_k = gamma * bytes_per_point * n_k * 8."""
    bpp = cfg["arrivals"]["bytes_per_point"]
    return np.array([gamma * float(n * bpp * 8) for n in points_per_agent])


def upward_rank(cost, succ):
    """rank(v) = cost(v) + max over successors w of rank(w) (0 without
    successors): the longest path from v to an exit, v's own cost included."""
    memo = {}

    def rank(v):
        if v not in memo:
            memo[v] = cost[v] + max((rank(w) for w in succ.get(v, ())), default=0)
        return memo[v]

    return {v: rank(v) for v in cost}


def dagrank_weights(c_enc_ns, c_post_ns):
    """omega_k of the profiled DAG: encoders E_k -> post-join chain P_1 ->
    ... -> P_m; omega_k = rank(E_k) / max_j rank(E_j)."""
    K = len(c_enc_ns)
    cost = {("E", k): int(c) for k, c in enumerate(c_enc_ns)}
    succ = {("E", k): [("P", 0)] for k in range(K)}
    for i, c in enumerate(c_post_ns):
        cost[("P", i)] = int(c)
        if i + 1 < len(c_post_ns):
            succ[("P", i)] = [("P", i + 1)]
    rk = upward_rank(cost, succ)
    top = max(rk[("E", k)] for k in range(K))
    return [float(rk[("E", k)]) / float(top) for k in range(K)]


def trial(R, B_bits, cfg, scheduler, c_enc_ns, c_post_ns):
    """One paired measured-DAG trial.  Returns dict(tau, feasible, a_ns,
    T_R, T_B, W_pre) with integer-nanosecond latencies (None if the frame
    is communication-infeasible)."""
    arr = cfg["arrivals"]
    K = cfg["K"]
    w = None
    if scheduler == "dagrank":
        w = dagrank_weights(c_enc_ns, c_post_ns)
    elif scheduler == "tw_maxrate":
        w = arr["task_weights"]
    pol = U.make_policy(scheduler, K, slot_s=arr["slot_s"], weights=w)
    res = U.emulate(R, B_bits, arr["slot_s"], pol)
    out = dict(tau=[int(v) for v in res["tau"]], feasible=res["feasible"], a_ns=None, T_R=None, T_B=None,
               W_pre=None)
    if res["feasible"]:
        slot_ns = int(round(arr["slot_s"] * 1e9))
        a = [int(v) * slot_ns for v in res["tau"]]
        TR, TB, W = S.paired_int(a, c_enc_ns, c_post_ns)
        out.update(a_ns=a, T_R=TR, T_B=TB, W_pre=W)
    return out
