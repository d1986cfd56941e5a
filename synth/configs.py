"""Workload descriptions of the five evaluated detector instances plus two
small parity instances.

Each entry states only data: agent count, point-cloud recipe, BEV region,
pillar size, network widths, precision, fusion kind, detection threshold
and the arrival-trace recipe.  The shapes follow the paper's fork-join
detector (Sec. V-A1: a PointPillars-based intermediate-fusion detector with
one shared encoder per agent); the concrete sizes are those of the five
synthetic workloads the implementation is measured on.

Grid sizes, layer shapes and every other derived quantity are computed by
the consumers (oracle and library) on their own.
"""

import copy
import math

# PointPillars car anchor (w, l, h, z-centre, yaws) used by both the oracle
# and the library's decode step.
_ANCHORS = dict(
    n_anchors=2,
    anchor_w=1.6,
    anchor_l=3.9,
    anchor_h=1.5,
    anchor_z=-1.0,
    anchor_yaws=(0.0, math.pi / 2.0),
)

# Rotated NMS after decoding: bird's-eye-view IoU threshold and the number of
# top-scoring decoded boxes that take part.
_NMS = dict(
    nms_iou_threshold=0.15,
    nms_max_candidates=4096,
)

_MIXTURE = dict(
    ground_frac=0.7,
    ground_z_mean=-1.7,
    ground_z_std=0.05,
    blob_points=200,
    blob_sigma=0.5,
    blob_zc=(-1.7, 0.0),
)

# Slot-level OFDMA uplink of the evaluation (Sec. V-A2, Table of simulation
# parameters): K = 6 mobile agents in an 80 x 50 m area with the edge server
# at its centre, F = 8 resource blocks, 1 ms slots, a 900-slot horizon and a
# 400 ms service deadline.  Reference rate of each agent-RB pair uniform in
# [250, 4500] kbit/s, scaled by distance attenuation (path-loss exponent
# 2.15), agent-specific blockage and per-slot, per-RB small-scale fading.
# Payloads scale by gamma, rates by beta; nominal point (1.0, 0.8).  The
# values the paper does not give (reference distance, speeds, blockage
# statistics, fading law) are this workload's own choices.
_OFDMA = dict(
    kind="ofdma",
    n_rb=8,
    slot_s=1e-3,
    t_max_slots=900,
    deadline_s=0.4,
    area_m=(80.0, 50.0),
    server_m=(40.0, 25.0),
    path_loss_exp=2.15,
    ref_distance_m=30.0,
    ref_rate_bps=(250e3, 4500e3),
    speed_mps=(5.0, 15.0),
    blockage_fraction=0.2,
    blockage_dwell_slots=200.0,
    blockage_loss_db=4.0,
    gammas=(0.5, 1.0, 1.5, 2.0),
    betas=(0.6, 0.8, 1.0, 1.2, 1.4),
    nominal=(1.0, 0.8),
    schedulers=("maxrate", "maxweight", "earliest_release", "dagrank", "tw_maxrate"),
    task_weights=(1.00, 0.80, 1.20, 0.70, 1.05, 0.60),
    bytes_per_point=16,
)

_PP_BACKBONE_64 = ((2, 64, 3), (2, 128, 5), (2, 256, 5))
_PP_BACKBONE_128 = ((2, 128, 3), (2, 256, 5), (2, 256, 5))

_CONFIGS = {
    # Tiny CPU-seconds instance: 2 agents, fp32, max fusion, fixed arrivals.
    "c1": dict(
        K=2,
        n_points=2000,
        dist="uniform",
        x_range=(-25.6, 25.6),
        y_range=(-25.6, 25.6),
        z_range=(-3.0, 1.0),
        pillar=0.8,
        max_pts=32,
        c_pfn=32,
        precision="fp32",
        stages=((1, 32, 2),),
        up_channels=0,
        fusion="max",
        logit_threshold=1.0,
        arrivals=dict(kind="fixed", a_ms=(0.0, 5.0)),
        traces=1,
        reps=50,
        seed_index=0,
    ),
    # Three-agent bf16 instance, max fusion, exponential arrival gaps.
    "c2": dict(
        K=3,
        n_points=20000,
        dist="mixture",
        x_range=(-51.2, 51.2),
        y_range=(-51.2, 51.2),
        z_range=(-3.0, 1.0),
        pillar=0.4,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=_PP_BACKBONE_64,
        up_channels=128,
        fusion="max",
        logit_threshold=0.8,
        arrivals=dict(kind="exp_gaps", mean_ms=10.0),
        traces=30,
        reps=5,
        seed_index=1,
    ),
    # Five-agent attention-fusion instance with uplink-driven arrivals.
    "c3": dict(
        K=5,
        n_points=40000,
        dist="mixture",
        x_range=(-70.4, 70.4),
        y_range=(-20.0, 20.0),
        z_range=(-3.0, 1.0),
        pillar=0.4,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=_PP_BACKBONE_64,
        up_channels=128,
        fusion="attn",
        logit_threshold=1.2,
        arrivals=dict(
            kind="uplink",
            snr_db=(10.0,),
            schedulers=("rr",),
            bandwidth_hz=20e6,
            slot_s=1e-3,
            n_rb=1,
            pf_window=100,
            bytes_per_pillar=64 * 2,
            t_max_slots=20000,
        ),
        traces=30,
        reps=5,
        seed_index=2,
    ),
    # Communication-load sweep on the config-3 network (same points and
    # weights as c3; only the arrival traces differ).
    "c4": dict(
        base="c3",
        arrivals=dict(
            kind="uplink",
            snr_db=(0.0, 10.0, 20.0),
            schedulers=("rr", "pf"),
            bandwidth_hz=20e6,
            slot_s=1e-3,
            n_rb=1,
            pf_window=100,
            bytes_per_pillar=64 * 2,
            t_max_slots=20000,
        ),
        traces=200,
        reps=3,
        seed_index=3,
    ),
    # Eight-agent stress instance, 512x512 BEV, attention fusion.
    "c5": dict(
        K=8,
        n_points=100000,
        dist="mixture",
        x_range=(-51.2, 51.2),
        y_range=(-51.2, 51.2),
        z_range=(-3.0, 1.0),
        pillar=0.2,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=_PP_BACKBONE_128,
        up_channels=128,
        fusion="attn",
        logit_threshold=1.2,
        arrivals=dict(kind="lognormal", median_ms=20.0, sigma=0.8),
        traces=30,
        reps=5,
        seed_index=4,
    ),
    # Small parity instances: grids whose stage sizes are ragged (44x60 ->
    # 22x30 -> 11x15 -> 6x8, upsampled x4 to 24x32 and cropped to 22x30),
    # so every GEMM has a partial tile and the x4 deconvolution crops.
    "t_max": dict(
        K=3,
        n_points=6000,
        dist="mixture",
        x_range=(-12.0, 12.0),
        y_range=(-8.8, 8.8),
        z_range=(-3.0, 1.0),
        pillar=0.4,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=((2, 64, 2), (2, 128, 2), (2, 256, 2)),
        up_channels=128,
        fusion="max",
        logit_threshold=0.8,
        arrivals=dict(kind="exp_gaps", mean_ms=2.0),
        traces=4,
        reps=2,
        seed_index=5,
    ),
    "t_attn": dict(
        K=4,
        n_points=6000,
        dist="mixture",
        x_range=(-12.0, 12.0),
        y_range=(-8.8, 8.8),
        z_range=(-3.0, 1.0),
        pillar=0.4,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=((2, 64, 2), (2, 128, 2), (2, 256, 2)),
        up_channels=128,
        fusion="attn",
        logit_threshold=1.5,
        arrivals=dict(kind="lognormal", median_ms=3.0, sigma=0.8),
        traces=4,
        reps=2,
        seed_index=6,
    ),
    # Conv-tiling instance: c5's channels (128 / 256 / 256) on an 88 x 120
    # grid, so every halo tiling and the implicit GEMM run on several tiles
    # with ragged edges (stage grids 44 x 60, 22 x 30, 11 x 15).
    "t_var": dict(
        K=2,
        n_points=12000,
        dist="mixture",
        x_range=(-17.6, 17.6),
        y_range=(-24.0, 24.0),
        z_range=(-3.0, 1.0),
        pillar=0.4,
        max_pts=32,
        c_pfn=64,
        precision="bf16",
        stages=((2, 128, 2), (2, 256, 2), (2, 256, 2)),
        up_channels=128,
        fusion="attn",
        logit_threshold=1.5,
        arrivals=dict(kind="lognormal", median_ms=3.0, sigma=0.8),
        traces=4,
        reps=2,
        seed_index=8,
    ),
}

# Six-agent measured-DAG instance: the config-3 network (bf16, attention
# fusion, 352 x 100 grid) with six agents whose branch inputs are 60.6 to
# 65.2 KiB of float32 points (16 bytes each; Sec. V-A1), sent over the OFDMA
# uplink above.
_CONFIGS["s6"] = dict(
    _CONFIGS["c3"],
    K=6,
    points_per_agent=(3878, 3937, 3996, 4055, 4114, 4173),
    n_points=4173,
    arrivals=_OFDMA,
    traces=30,
    reps=3,
    seed_index=7,
)

CONFIG_NAMES = ("c1", "c2", "c3", "c4", "c5", "t_max", "t_attn", "t_var", "s6")

ROOT_SEED = 20260830


def config(name):
    """Return a fully populated copy of the named workload description."""
    if name not in _CONFIGS:
        raise KeyError("unknown config %r" % (name,))
    raw = _CONFIGS[name]
    if "base" in raw:
        cfg = copy.deepcopy(_CONFIGS[raw["base"]])
        cfg.update(copy.deepcopy({k: v for k, v in raw.items() if k != "base"}))
        cfg["data_from"] = raw["base"]
    else:
        cfg = copy.deepcopy(raw)
        cfg["data_from"] = name
    cfg["name"] = name
    cfg.update(copy.deepcopy(_ANCHORS))
    cfg.update(copy.deepcopy(_NMS))
    if cfg.get("dist") == "mixture":
        cfg["mixture"] = dict(_MIXTURE)
    return cfg


def network_layers(cfg):
    """Ordered weight tensors of the network: (name, shape, fan_in).

    Order and shapes are the canonical weight order of the library's flat
    weight blob as well:
      pfn_w [4, C_pfn], pfn_b [C_pfn]
      per stage s, conv l: s{s}c{l}_w [3, 3, C_in, C_out] (HWIO), _b [C_out]
      per stage s (if up_channels): up{s}_w [u, u, C_s, up] with u = 2**s
                                    relative to stage 0, up{s}_b [up]
      head_w [C, 2 * 8], head_b [2 * 8]
    """
    out = []
    c_pfn = cfg["c_pfn"]
    out.append(("pfn_w", (4, c_pfn), 4))
    out.append(("pfn_b", (c_pfn,), None))
    c_in = c_pfn
    stage_out = []
    for s, (stride, c_out, n_convs) in enumerate(cfg["stages"]):
        for l in range(n_convs):
            cin_l = c_in if l == 0 else c_out
            out.append(("s%dc%d_w" % (s, l), (3, 3, cin_l, c_out), 9 * cin_l))
            out.append(("s%dc%d_b" % (s, l), (c_out,), None))
        c_in = c_out
        stage_out.append(c_out)
    up = cfg["up_channels"]
    if up:
        rel = 1
        for s, (stride, c_out, _n) in enumerate(cfg["stages"]):
            if s > 0:
                rel *= stride
            out.append(("up%d_w" % s, (rel, rel, c_out, up), c_out))
            out.append(("up%d_b" % s, (up,), None))
        c_head = up * len(cfg["stages"])
    else:
        c_head = stage_out[-1]
    n_out = cfg["n_anchors"] * 8
    out.append(("head_w", (c_head, n_out), c_head))
    out.append(("head_b", (n_out,), None))
    return out
