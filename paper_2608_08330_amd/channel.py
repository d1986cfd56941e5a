"""OFDMA uplink channel of the evaluation (harness layer).

Turns the seeded draws of one channel trace (``synth.ofdma_draws``) into
the per-slot rate of every agent-RB pair, R[t, k, f] in bit/s, for the
slot-level uplink emulation (Sec. V-A2: K agents moving in a W x H area
around a central edge server, F RBs of 1 ms slots, reference rate per
agent-RB pair, distance attenuation with exponent alpha, agent-specific
blockage, slot-level RB-dependent small-scale fading, bandwidth scale beta;
payloads scale by gamma):

  R[t, k, f] = beta * Rref[k, f] * G(d_k[t]) * Z_k[t] * h[t, k, f]

  * rates scale linearly with the channel power gain (low-SNR regime);
  * d_k[t]: distance to the server at the start of slot t, positions moving
    straight at constant speed and reflecting at the area walls;
  * G(d) = min(1, (d_ref / d)^alpha);
  * Z_k[t] = 10^(-L_b / 10) while agent k is blocked, else 1; blockage is a
    two-state chain per agent (blocked in slot 1 iff u0 < rho; a blocked
    agent clears iff u < 1 / D, a clear one becomes blocked iff
    u < rho / ((1 - rho) D), D the mean blocked dwell in slots, rho the
    long-run blocked fraction);
  * h ~ Exp(1) i.i.d. per agent, RB and slot.
"""

import math

import numpy as np


def positions(draw, arr):
    """[T, K] x and y (m) at the start of every slot."""
    T = arr["t_max_slots"]
    tau = np.arange(T, dtype=np.int64) * arr["slot_s"]
    vx = np.array([v * math.cos(h) for v, h in zip(draw["speed_mps"], draw["heading"])])
    vy = np.array([v * math.sin(h) for v, h in zip(draw["speed_mps"], draw["heading"])])
    out = []
    for axis, v, L in ((0, vx, arr["area_m"][0]), (1, vy, arr["area_m"][1])):
        p = draw["pos0_m"][:, axis][None, :] + v[None, :] * tau[:, None]
        u = np.mod(p, 2.0 * L)
        out.append(np.where(u <= L, u, 2.0 * L - u))
    return out[0], out[1]


def path_gains(draw, arr):
    """[T, K] G(d_k[t]).  hypot and pow come from the C library (math), one
    value at a time, so that the gains are correctly rounded the same way
    wherever they are evaluated."""
    x, y = positions(draw, arr)
    sx, sy = arr["server_m"]
    d_ref, alpha = arr["ref_distance_m"], arr["path_loss_exp"]
    g = np.empty(x.shape)
    for i, (px, py) in enumerate(zip((x - sx).ravel().tolist(), (y - sy).ravel().tolist())):
        d = math.hypot(px, py)
        g.flat[i] = (d_ref / d) ** alpha if d > d_ref else 1.0
    return g


def blocked(draw, arr):
    """[T, K] bool blockage state per slot."""
    T = arr["t_max_slots"]
    rho, D = arr["blockage_fraction"], arr["blockage_dwell_slots"]
    p_clear = 1.0 / D
    p_block = rho / ((1.0 - rho) * D)
    u = draw["block_u"]
    st = np.empty(u.shape, dtype=bool)
    st[0] = draw["block_u0"] < rho
    for t in range(1, T):
        st[t] = np.where(st[t - 1], ~(u[t] < p_clear), u[t] < p_block)
    return st


def rates(draw, cfg, beta):
    """[T, K, F] float64 rates in bit/s of one trace at bandwidth scale beta."""
    arr = cfg["arrivals"]
    g = path_gains(draw, arr)
    z = np.where(blocked(draw, arr), 10.0 ** (-arr["blockage_loss_db"] / 10.0), 1.0)
    R = (beta * draw["ref_rate_bps"])[None, :, :] * g[:, :, None]
    R = R * z[:, :, None]
    return R * draw["fading"]


def payload_bits(cfg, points_per_agent, gamma):
    """B_k = gamma * (bytes of agent k's float32 points) * 8."""
    bpp = cfg["arrivals"]["bytes_per_point"]
    return np.array([gamma * float(int(n) * bpp * 8) for n in points_per_agent])
