"""Pins of the oracle's pillarization (cell index, grouping, 32-point cap)
and bfloat16 rounding, against brute force, exact rational geometry and a
library conversion."""

from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import network as N
from oracle.bf16 import round_bf16


def _cfg():
    return synth.config("c1")  # 64 x 64 grid, 0.8 m pillars, [-25.6, 25.6)^2 x [-3, 1)


# ---------------------------------------------------------------- bf16

def test_bf16_matches_torch_on_float32_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-30, 30, 200000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_ties_to_even_and_fixed_points():
    one = 1.0
    half_ulp = 2.0 ** -8  # bf16 spacing at 1 is 2^-7
    # exactly halfway between 1 and 1 + 2^-7: even significand is 1
    assert round_bf16(np.array([one + half_ulp]))[0] == 1.0
    # halfway between 1 + 2^-7 and 1 + 2^-6: even significand is 1 + 2^-6
    assert round_bf16(np.array([one + 3 * half_ulp]))[0] == 1.0 + 2.0 ** -6
    # just above halfway rounds up
    assert round_bf16(np.array([one + half_ulp + 2.0 ** -30]))[0] == 1.0 + 2.0 ** -7
    vals = np.array([0.0, -2.0, 0.5, 3.0, 1.0 + 2.0 ** -7, -(2.0 ** -120)])
    assert np.array_equal(round_bf16(vals), vals)


# ---------------------------------------------------------------- cell ids

def _geom_cell(p, cfg):
    """Exact rational containment: the cell whose closed-open box holds the
    point, or -1 (no floating point involved)."""
    H, W = N.grid(cfg)
    if not np.all(np.isfinite(p)):
        return -1
    x, y, z = (Fraction(float(v)) for v in p[:3])
    x0, x1 = (Fraction(float(np.float32(v))) for v in cfg["x_range"])
    y0, y1 = (Fraction(float(np.float32(v))) for v in cfg["y_range"])
    z0, z1 = (Fraction(float(np.float32(v))) for v in cfg["z_range"])
    if not (x0 <= x < x1 and y0 <= y < y1 and z0 <= z < z1):
        return -1
    v = Fraction(float(np.float32(cfg["pillar"])))
    ix = int((x - x0) // v)
    iy = int((y - y0) // v)
    if not (0 <= ix < W and 0 <= iy < H):
        return -1
    return iy * W + ix


def _near_edge(p, cfg, eps=1e-4):
    v = float(np.float32(cfg["pillar"]))
    fx = (float(p[0]) - float(np.float32(cfg["x_range"][0]))) / v
    fy = (float(p[1]) - float(np.float32(cfg["y_range"][0]))) / v
    return min(abs(fx - round(fx)), abs(fy - round(fy))) < eps


def test_cell_ids_match_exact_geometry_away_from_edges():
    cfg = _cfg()
    rng = np.random.default_rng(7)
    pts = np.empty((3000, 4), dtype=np.float32)
    pts[:, 0] = rng.uniform(-27, 27, 3000)
    pts[:, 1] = rng.uniform(-27, 27, 3000)
    pts[:, 2] = rng.uniform(-3.5, 1.5, 3000)
    pts[:, 3] = rng.uniform(0, 1, 3000)
    cell = N.cell_ids(pts, cfg)
    checked = 0
    for i in range(len(pts)):
        if _near_edge(pts[i], cfg):
            continue
        assert cell[i] == _geom_cell(pts[i], cfg), i
        checked += 1
    assert checked > 2500


def test_cell_ids_special_points():
    cfg = _cfg()
    H, W = N.grid(cfg)
    assert (H, W) == (64, 64)
    pts = np.array([
        [0.0, 0.0, 0.0, 0.5],          # centre: 25.6f = 32 * 0.8f exactly -> (32, 32)
        [-25.6, -25.6, -3.0, 0.0],     # lower corner, inclusive -> cell 0
        [25.6, 0.0, 0.0, 0.0],         # x = xmax excluded
        [0.0, 25.6, 0.0, 0.0],         # y = ymax excluded
        [0.0, 0.0, 1.0, 0.0],          # z = zmax excluded
        [0.0, 0.0, -3.0, 0.0],         # z = zmin included
        [np.nan, 0.0, 0.0, 0.0],       # non-finite coordinate
        [0.0, 0.0, 0.0, np.inf],       # non-finite intensity
        [np.inf, 0.0, 0.0, 0.0],
        [-25.7, 0.0, 0.0, 0.0],        # left of the region
    ], dtype=np.float32)
    cell = N.cell_ids(pts, cfg)
    assert cell.tolist() == [32 * 64 + 32, 0, -1, -1, -1, 32 * 64 + 32, -1, -1, -1, -1]


def test_largest_float_below_xmax_stays_in_grid():
    cfg = _cfg()
    x = np.nextafter(np.float32(25.6), np.float32(0))
    cell = N.cell_ids(np.array([[x, x, 0, 0]], dtype=np.float32), cfg)
    H, W = N.grid(cfg)
    assert 0 <= cell[0] < H * W
    assert cell[0] % W == W - 1 and cell[0] // W == H - 1


# ---------------------------------------------------------------- grouping

def _brute_pillars(cell, cap):
    groups = {}
    for i, c in enumerate(cell.tolist()):
        if c >= 0:
            groups.setdefault(c, []).append(i)
    cells = sorted(groups)
    return cells, [len(groups[c]) for c in cells], [groups[c][:cap] for c in cells]


def test_pillars_brute_force_and_conservation():
    cfg = synth.config("t_max")
    fr = synth.make_frame(cfg)
    biggest = 0
    for pts in fr["points"]:
        cell = N.cell_ids(pts, cfg)
        pil = N.pillars(cell, 32)
        cells, counts, used = _brute_pillars(cell, 32)
        assert pil["cells"].tolist() == cells
        assert pil["counts"].tolist() == counts
        assert [u.tolist() for u in pil["used"]] == used
        assert int(pil["counts"].sum()) == int((cell >= 0).sum())
        assert np.all(np.diff(pil["cells"]) > 0)
        biggest = max(biggest, max(counts))
    assert biggest > 32  # the cap is exercised by this workload


def test_pillar_cap_keeps_lowest_indices():
    cfg = _cfg()
    rng = np.random.default_rng(3)
    pts = np.zeros((150, 4), dtype=np.float32)
    pts[:, :2] = rng.uniform(-25.6, 25.6, (150, 2))
    sel = rng.choice(150, 100, replace=False)
    pts[sel, 0] = 0.3
    pts[sel, 1] = 0.3
    cell = N.cell_ids(pts, cfg)
    pil = N.pillars(cell, 32)
    c = int(cell[sel[0]])
    p = pil["cells"].tolist().index(c)
    assert pil["counts"][p] == 100 + int(np.sum(cell[np.setdiff1d(np.arange(150), sel)] == c))
    members = np.nonzero(cell == c)[0]
    assert pil["used"][p].tolist() == sorted(members.tolist())[:32]


def test_pillars_empty_and_all_invalid():
    pil = N.pillars(np.zeros(0, dtype=np.int64), 32)
    assert len(pil["cells"]) == 0
    pil = N.pillars(np.full(5, -1), 32)
    assert len(pil["cells"]) == 0 and pil["counts"].sum() == 0
