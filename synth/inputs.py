"""Seeded random draws: point clouds, agent poses, network weights, arrival
vectors and per-slot fading gains.

Seeding: ``SeedSequence(ROOT_SEED).spawn(9)[cfg['seed_index']]`` is the
config's sequence; it spawns four children, in this order, for points,
poses, weights and arrival traces.  A config whose data comes from another
config (the load sweep reuses the config-3 network and frames) takes the
points, poses and weights children of that config and only its own trace
child.  All generators use numpy's PCG64.
"""

import math

import numpy as np

from .configs import ROOT_SEED, config, network_layers

_N_CONFIG_SEEDS = 9
_CHILD = {"points": 0, "poses": 1, "weights": 2, "traces": 3}

# Standard deviation of the bias vectors.  The weight matrices are He-normal
# (variance 2 / fan_in); biases are small and non-zero so that every bias
# epilogue is exercised by the end-to-end parity checks.
BIAS_STD = 0.1


def seed_children(cfg, what):
    """SeedSequence for one kind of draw of a config."""
    src = cfg if what == "traces" else config(cfg["data_from"])
    root = np.random.SeedSequence(ROOT_SEED).spawn(_N_CONFIG_SEEDS)[src["seed_index"]]
    return root.spawn(4)[_CHILD[what]]


def _rng(cfg, what, *sub):
    ss = seed_children(cfg, what)
    for s in sub:
        ss = ss.spawn(s + 1)[s]
    return np.random.Generator(np.random.PCG64(ss))


def _uniform_cloud(rng, n, cfg):
    x0, x1 = cfg["x_range"]
    y0, y1 = cfg["y_range"]
    z0, z1 = cfg["z_range"]
    pts = np.empty((n, 4), dtype=np.float64)
    pts[:, 0] = rng.uniform(x0, x1, n)
    pts[:, 1] = rng.uniform(y0, y1, n)
    pts[:, 2] = rng.uniform(z0, z1, n)
    pts[:, 3] = rng.uniform(0.0, 1.0, n)
    return pts


def _mixture_cloud(rng, n, cfg):
    mx = cfg["mixture"]
    x0, x1 = cfg["x_range"]
    y0, y1 = cfg["y_range"]
    n_ground = int(round(mx["ground_frac"] * n))
    n_blob = n - n_ground
    ground = np.empty((n_ground, 4))
    ground[:, 0] = rng.uniform(x0, x1, n_ground)
    ground[:, 1] = rng.uniform(y0, y1, n_ground)
    ground[:, 2] = rng.normal(mx["ground_z_mean"], mx["ground_z_std"], n_ground)
    ground[:, 3] = rng.uniform(0.0, 1.0, n_ground)
    per = mx["blob_points"]
    n_blobs = int(math.ceil(n_blob / per)) if n_blob else 0
    centres = np.empty((n_blobs, 3))
    centres[:, 0] = rng.uniform(x0, x1, n_blobs)
    centres[:, 1] = rng.uniform(y0, y1, n_blobs)
    centres[:, 2] = rng.uniform(mx["blob_zc"][0], mx["blob_zc"][1], n_blobs)
    owner = np.repeat(np.arange(n_blobs), per)[:n_blob]
    blob = np.empty((n_blob, 4))
    blob[:, :3] = centres[owner] + rng.normal(0.0, mx["blob_sigma"], (n_blob, 3))
    blob[:, 3] = rng.uniform(0.0, 1.0, n_blob)
    pts = np.concatenate([ground, blob], axis=0)
    # Interleave ground and object returns so that point order is not
    # correlated with position.
    return pts[rng.permutation(n)]


def points_per_agent(cfg):
    """Point count of every agent's cloud (``points_per_agent`` if the
    workload lists one per agent, else ``n_points`` each)."""
    n = cfg.get("points_per_agent")
    return [int(v) for v in n] if n is not None else [int(cfg["n_points"])] * cfg["K"]


def make_points(cfg, frame=0):
    """List of K float32 arrays [n_k, 4] = (x, y, z, intensity), agent frame.
    Frame f > 0 of a stream draws from its own child sequences (frame 0 is
    the config's frame)."""
    out = []
    for k, n in enumerate(points_per_agent(cfg)):
        rng = _rng(cfg, "points", k) if frame == 0 else _rng(cfg, "points", k, frame)
        if cfg["dist"] == "uniform":
            pts = _uniform_cloud(rng, n, cfg)
        elif cfg["dist"] == "mixture":
            pts = _mixture_cloud(rng, n, cfg)
        else:
            raise ValueError(cfg["dist"])
        out.append(np.ascontiguousarray(pts.astype(np.float32)))
    return out


def make_poses(cfg, frame=0):
    """[K, 3] float64 agent-to-ego poses (yaw rad, tx m, ty m).

    Agent 0 is the ego vehicle (identity).  Other agents draw yaw uniform in
    [-pi, pi) and a translation uniform in [-5, 5) m per axis.  Frame f > 0
    of a stream draws from its own child sequence.
    """
    rng = _rng(cfg, "poses") if frame == 0 else _rng(cfg, "poses", frame)
    K = cfg["K"]
    poses = np.zeros((K, 3), dtype=np.float64)
    if K > 1:
        poses[1:, 0] = rng.uniform(-math.pi, math.pi, K - 1)
        poses[1:, 1:] = rng.uniform(-5.0, 5.0, (K - 1, 2))
    return poses


def make_weights(cfg):
    """Dict name -> float32 array.  Weight matrices He-normal, biases small."""
    rng = _rng(cfg, "weights")
    w = {}
    for name, shape, fan_in in network_layers(cfg):
        if fan_in is None:
            arr = rng.normal(0.0, BIAS_STD, shape)
        else:
            arr = rng.normal(0.0, math.sqrt(2.0 / fan_in), shape)
        w[name] = np.ascontiguousarray(arr.astype(np.float32))
    return w


def make_frame(name_or_cfg, frame=0):
    """Inputs of one frame: points, poses and the (frame-independent)
    weights.  ``frame`` > 0 gives further frames of a stream: new points and
    poses, the same network."""
    cfg = config(name_or_cfg) if isinstance(name_or_cfg, str) else name_or_cfg
    return dict(
        cfg=cfg,
        points=make_points(cfg, frame),
        poses=make_poses(cfg, frame),
        weights=make_weights(cfg),
    )


def arrival_draws(cfg, n_traces=None):
    """Arrival vectors in ms, [n_traces, K], for configs whose arrivals are
    drawn directly (fixed, exponential gaps, log-normal).

    Exponential gaps: K i.i.d. gaps with the configured mean; the j-th
    smallest arrival time is the sum of the first j gaps and is given to
    agent perm[j] of a seeded permutation, so arrival order is not index
    order.  Log-normal: each agent's completion time is exp(N(ln median,
    sigma^2)) ms, i.i.d.
    """
    arr = cfg["arrivals"]
    K = cfg["K"]
    n = cfg["traces"] if n_traces is None else n_traces
    if arr["kind"] == "fixed":
        return np.tile(np.asarray(arr["a_ms"], dtype=np.float64), (n, 1))
    out = np.empty((n, K), dtype=np.float64)
    for t in range(n):
        rng = _rng(cfg, "traces", t)
        if arr["kind"] == "exp_gaps":
            gaps = rng.exponential(arr["mean_ms"], K)
            perm = rng.permutation(K)
            times = np.cumsum(gaps)
            out[t, perm] = times
        elif arr["kind"] == "lognormal":
            out[t] = np.exp(rng.normal(math.log(arr["median_ms"]), arr["sigma"], K))
        else:
            raise ValueError("arrivals of kind %r come from the uplink model" % arr["kind"])
    return out


def fading_draws(cfg, trace, n_slots=None):
    """Per-slot, per-agent, per-RB small-scale power gains |h|^2 ~ Exp(1),
    float64 [n_slots, K, n_rb], i.i.d.  The same draws serve every
    (SNR, scheduler) setting of a trace, so settings are compared on common
    channel realizations."""
    arr = cfg["arrivals"]
    n_slots = arr["t_max_slots"] if n_slots is None else n_slots
    rng = _rng(cfg, "traces", trace)
    return rng.exponential(1.0, (n_slots, cfg["K"], arr["n_rb"]))


def ofdma_draws(cfg, trace):
    """Random draws of one OFDMA channel trace (T = t_max_slots slots, K
    agents, F = n_rb RBs), independent of the payload and bandwidth scales
    and of the scheduler, so that every (gamma, beta, scheduler) cell of a
    trace sees the same channel realisation:

      ref_rate_bps [K, F]  reference rate of each agent-RB pair, uniform
                           in ref_rate_bps
      pos0_m       [K, 2]  start position, uniform over the area
      heading      [K]     direction of travel, uniform in [-pi, pi)
      speed_mps    [K]     speed, uniform in speed_mps
      block_u0     [K]     uniform [0, 1): initial blockage draw
      block_u      [T, K]  uniform [0, 1): per-slot blockage transition draws
      fading       [T, K, F] small-scale power gains, Exp(1) i.i.d.
    """
    arr = cfg["arrivals"]
    T, K, F = arr["t_max_slots"], cfg["K"], arr["n_rb"]
    rng = _rng(cfg, "traces", trace)
    lo, hi = arr["ref_rate_bps"]
    out = dict(ref_rate_bps=rng.uniform(lo, hi, (K, F)))
    out["pos0_m"] = np.stack([rng.uniform(0.0, arr["area_m"][0], K), rng.uniform(0.0, arr["area_m"][1], K)], axis=1)
    out["heading"] = rng.uniform(-math.pi, math.pi, K)
    out["speed_mps"] = rng.uniform(arr["speed_mps"][0], arr["speed_mps"][1], K)
    out["block_u0"] = rng.uniform(0.0, 1.0, K)
    out["block_u"] = rng.uniform(0.0, 1.0, (T, K))
    out["fading"] = rng.exponential(1.0, (T, K, F))
    return out
