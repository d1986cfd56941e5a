"""The pillar sort at sizes off the common path, bit-exact against the
oracle (pillar cells, counts and the points each pillar feeds to the
point-feature net): an agent with three agents' clouds (586 point blocks
over 128 tiles of cells), and an agent with 15,000,000 points on 4,096
cells, where each of the two tiles holds far more points than the tile
sort keeps in registers and every pillar is over the cap."""

import sys

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R
from tests.helpers import check_members, make_ctx, run_frame

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _check_pillars(ctx, cfg, points, agent):
    pil = N.pillars(N.cell_ids(points, cfg), cfg["max_pts"])
    cells = R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_CELLS, agent, np.int32)
    counts = R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_COUNTS, agent, np.int32)
    assert np.array_equal(cells, pil["cells"].astype(np.int32)), agent
    assert np.array_equal(counts, pil["counts"].astype(np.int32)), agent
    check_members(ctx, cfg, points, agent)


def test_many_point_blocks_over_many_tiles():
    # c5 geometry (128 tiles); agent 0 holds three agents' clouds, 586 point
    # blocks
    cfg = synth.config("c5")
    fr = synth.make_frame(cfg)
    big = np.ascontiguousarray(np.concatenate(fr["points"][:3]))
    fr["points"] = [big] + fr["points"][1:]
    _say("c5 with %d points in agent 0" % len(big))
    with make_ctx(cfg, fr, max_points=len(big)) as ctx:
        run_frame(ctx, fr)
        _check_pillars(ctx, cfg, big, 0)
        _check_pillars(ctx, cfg, fr["points"][1], 1)


def test_fifteen_million_points_on_two_tiles():
    # c1 geometry (2 tiles of cells, 4,096 cells); 15,000,000 points in
    # agent 0: 29,297 point blocks, 7.5 million points per tile
    cfg = synth.config("c1")
    fr = synth.make_frame(cfg)
    n = 15_000_000
    rng = np.random.default_rng(11)
    big = np.empty((n, 4), np.float32)
    big[:, 0] = rng.uniform(cfg["x_range"][0], cfg["x_range"][1], n)
    big[:, 1] = rng.uniform(cfg["y_range"][0], cfg["y_range"][1], n)
    big[:, 2] = rng.uniform(cfg["z_range"][0], cfg["z_range"][1], n)
    big[:, 3] = rng.uniform(0.0, 1.0, n)
    fr["points"] = [big] + fr["points"][1:]
    _say("c1 with %d points in agent 0" % n)
    with make_ctx(cfg, fr, max_points=n) as ctx:
        run_frame(ctx, fr)
        _check_pillars(ctx, cfg, big, 0)
        _check_pillars(ctx, cfg, fr["points"][1], 1)
