"""Seeded synthetic inputs for the RTCC fork-join detector.

This package is the only code shared by the oracle (``oracle/``) and the
HIP path (``paper_2608_08330_amd/``).  It draws random numbers and states
workload shapes; it holds none of the method's arithmetic (no pillarization,
no network, no warp, no schedule, no uplink accounting).
"""

from .configs import CONFIG_NAMES, ROOT_SEED, config, network_layers
from .inputs import (
    make_points,
    make_poses,
    make_weights,
    make_frame,
    arrival_draws,
    fading_draws,
    ofdma_draws,
    points_per_agent,
    seed_children,
)

__all__ = [
    "CONFIG_NAMES",
    "config",
    "ROOT_SEED",
    "network_layers",
    "make_points",
    "make_poses",
    "make_weights",
    "make_frame",
    "arrival_draws",
    "fading_draws",
    "ofdma_draws",
    "points_per_agent",
    "seed_children",
]
