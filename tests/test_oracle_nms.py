"""Pins of the rotated-NMS oracle (oracle/nms.py) against closed forms,
brute force and invariants that a mistake in it would break."""

import math

import numpy as np
import pytest

from oracle import nms as O


def box(x, y, w, l, yaw, z=0.0, h=1.5):
    return np.array([x, y, z, w, l, h, yaw], dtype=np.float64)


def aligned_overlap(a, b):
    """Closed form for footprints whose sides are parallel to the axes
    (yaw a multiple of pi/2)."""
    def extent(bx):
        swap = int(round(bx[6] / (math.pi / 2))) % 2 == 1
        ex, ey = (bx[3], bx[4]) if swap else (bx[4], bx[3])  # l along x at yaw 0
        return bx[0] - ex / 2, bx[0] + ex / 2, bx[1] - ey / 2, bx[1] + ey / 2
    ax0, ax1, ay0, ay1 = extent(a)
    bx0, bx1, by0, by1 = extent(b)
    ix = max(0.0, min(ax1, bx1) - max(ax0, bx0))
    iy = max(0.0, min(ay1, by1) - max(ay0, by0))
    inter = ix * iy
    return inter / (a[3] * a[4] + b[3] * b[4] - inter)


def raster_intersection(a, b, n=1200):
    """Brute force: count sample points (cell centres of an n x n grid over
    the two boxes' bounding square) inside both footprints."""
    ca, cb = O.corners(a), O.corners(b)
    xs = [p[0] for p in ca + cb]
    ys = [p[1] for p in ca + cb]
    x0, x1, y0, y1 = min(xs), max(xs), min(ys), max(ys)
    gx = x0 + (np.arange(n) + 0.5) * (x1 - x0) / n
    gy = y0 + (np.arange(n) + 0.5) * (y1 - y0) / n
    X, Y = np.meshgrid(gx, gy)

    def inside(c):
        m = np.ones_like(X, dtype=bool)
        for i in range(4):
            p, q = c[i], c[(i + 1) % 4]
            m &= (q[0] - p[0]) * (Y - p[1]) - (q[1] - p[1]) * (X - p[0]) >= 0
        return m
    cell = (x1 - x0) * (y1 - y0) / (n * n)
    return float(np.sum(inside(ca) & inside(cb))) * cell


def test_identical_disjoint_contained():
    a = box(1.0, 2.0, 1.6, 3.9, 0.3)
    assert O.iou(a, a) == pytest.approx(1.0, abs=1e-12)
    assert O.iou(a, box(20.0, 2.0, 1.6, 3.9, 0.3)) == 0.0
    big = box(0.0, 0.0, 4.0, 6.0, 0.7)
    small = box(0.1, -0.2, 1.0, 2.0, 0.7)  # same heading, well inside
    assert O.iou(big, small) == pytest.approx(2.0 / 24.0, abs=1e-12)


def test_axis_aligned_closed_form():
    rng = np.random.default_rng(5)
    for _ in range(200):
        a = box(*rng.uniform(-2, 2, 2), *rng.uniform(0.5, 4, 2), rng.integers(0, 4) * math.pi / 2)
        b = box(*rng.uniform(-2, 2, 2), *rng.uniform(0.5, 4, 2), rng.integers(0, 4) * math.pi / 2)
        assert O.iou(a, b) == pytest.approx(aligned_overlap(a, b), abs=1e-12)


def test_shared_edges_closed_form():
    # integer positions and sizes with yaw a multiple of pi/2: edges of the
    # two footprints often lie on the same line (coincident up to the
    # rounding of cos / sin), the degenerate case of the clipping
    rng = np.random.default_rng(8)
    for _ in range(3000):
        a = box(*rng.integers(-3, 3, 2).astype(float), *rng.integers(1, 4, 2).astype(float),
                rng.integers(0, 4) * math.pi / 2)
        b = box(*rng.integers(-3, 3, 2).astype(float), *rng.integers(1, 4, 2).astype(float),
                rng.integers(0, 4) * math.pi / 2)
        assert O.iou(a, b) == pytest.approx(aligned_overlap(a, b), abs=1e-12)
    # contained with three shared sides
    a = box(1.0, 1.0, 2.0, 1.0, 3 * math.pi / 2)
    b = box(1.0, 0.0, 3.0, 2.0, math.pi)
    assert O.iou(a, b) == pytest.approx(1.0 / 3.0, abs=1e-12)


def test_square_rotated_45_degrees_is_an_octagon():
    # same centre, side s: the intersection is a regular octagon of inradius
    # s / 2, area 8 (s/2)^2 tan(pi/8) = 2 (sqrt 2 - 1) s^2
    s = 2.5
    inter = 2.0 * (math.sqrt(2.0) - 1.0) * s * s
    a, b = box(3.0, -1.0, s, s, 0.0), box(3.0, -1.0, s, s, math.pi / 4)
    assert O.intersection_area(O.corners(a), O.corners(b)) == pytest.approx(inter, rel=1e-12)
    assert O.iou(a, b) == pytest.approx(inter / (2 * s * s - inter), rel=1e-12)


def test_matches_rasterized_area():
    rng = np.random.default_rng(11)
    for _ in range(6):
        a = box(0.0, 0.0, *rng.uniform(1, 3, 2), rng.uniform(-math.pi, math.pi))
        b = box(*rng.uniform(-1, 1, 2), *rng.uniform(1, 3, 2), rng.uniform(-math.pi, math.pi))
        exact = O.intersection_area(O.corners(a), O.corners(b))
        # grid error is of the order of the boundary length times the cell size
        assert exact == pytest.approx(raster_intersection(a, b), abs=0.02 * min(a[3] * a[4], b[3] * b[4]))


def test_symmetry_and_rigid_motion_invariance():
    rng = np.random.default_rng(3)
    for _ in range(100):
        a = box(*rng.uniform(-1, 1, 2), *rng.uniform(0.5, 3, 2), rng.uniform(-math.pi, math.pi))
        b = box(*rng.uniform(-1, 1, 2), *rng.uniform(0.5, 3, 2), rng.uniform(-math.pi, math.pi))
        v = O.iou(a, b)
        assert O.iou(b, a) == pytest.approx(v, abs=1e-12)
        th, t = rng.uniform(-math.pi, math.pi), rng.uniform(-10, 10, 2)
        c, s = math.cos(th), math.sin(th)

        def move(bx):
            m = bx.copy()
            m[0], m[1] = c * bx[0] - s * bx[1] + t[0], s * bx[0] + c * bx[1] + t[1]
            m[6] = bx[6] + th
            return m
        assert O.iou(move(a), move(b)) == pytest.approx(v, abs=1e-12)
        # a half turn maps the rectangle onto itself
        a2 = a.copy()
        a2[6] += math.pi
        assert O.iou(a2, b) == pytest.approx(v, abs=1e-12)


def test_invalid_boxes_overlap_nothing():
    a = box(0.0, 0.0, 1.6, 3.9, 0.0)
    for bad in (box(np.nan, 0, 1.6, 3.9, 0), box(0, 0, np.inf, 3.9, 0), box(0, 0, 0.0, 3.9, 0),
                box(0, 0, 1.6, -1.0, 0), box(0, 0, 1.6, 3.9, np.nan)):
        assert O.iou(a, bad) == 0.0 and O.iou(bad, a) == 0.0


def test_nms_chain_keeps_the_far_end():
    # A overlaps B, B overlaps C, A and C apart; A ranks first: B is
    # suppressed, so C survives
    A, B, C = box(0, 0, 2, 4, 0), box(2.0, 0, 2, 4, 0), box(4.0, 0, 2, 4, 0)
    assert O.iou(A, B) > 0.3 and O.iou(B, C) > 0.3 and O.iou(A, C) == 0.0
    kept = O.nms([A, B, C], [0.9, 0.8, 0.7], [10, 11, 12], 0.15, 100)
    assert kept == [0, 2]
    # with B first, both neighbours go
    assert O.nms([A, B, C], [0.8, 0.9, 0.7], [10, 11, 12], 0.15, 100) == [1]


def test_nms_ties_threshold_and_candidate_cap():
    a = box(0, 0, 2, 4, 0)
    # equal scores: the lower anchor index ranks first
    assert O.nms([a, a], [0.5, 0.5], [7, 3], 0.15, 10) == [1]
    # IoU 1 is not above a threshold of 1: nothing is suppressed
    assert O.nms([a, a], [0.5, 0.6], [1, 2], 1.0, 10) == [0, 1]
    # strictly greater: IoU exactly at the threshold keeps the box
    b = box(2.0, 0, 2, 4, 0)  # overlap 2 x 2 of two 8 m^2 boxes: IoU = 4 / 12
    assert O.nms([a, b], [0.9, 0.8], [0, 1], 4.0 / 12.0 + 1e-12, 10) == [0, 1]
    assert O.nms([a, b], [0.9, 0.8], [0, 1], 4.0 / 12.0 - 1e-12, 10) == [0]
    # only the first max_candidates of the ranking take part
    far = [box(10.0 * i, 0, 2, 4, 0) for i in range(5)]
    assert O.nms(far, [0.1, 0.5, 0.3, 0.9, 0.2], [0, 1, 2, 3, 4], 0.15, 2) == [1, 3]
    # output in ascending anchor index
    assert O.nms(far, [0.1, 0.5, 0.3, 0.9, 0.2], [9, 8, 7, 6, 5], 0.15, 5) == [4, 3, 2, 1, 0]


def test_nms_result_is_a_valid_greedy_suppression():
    rng = np.random.default_rng(17)
    n = 150
    boxes = np.stack([box(*rng.uniform(-8, 8, 2), *rng.uniform(1, 2.5, 2), rng.uniform(-math.pi, math.pi))
                      for _ in range(n)])
    scores = rng.uniform(0, 1, n)
    aidx = rng.permutation(1000)[:n]
    thr = 0.15
    kept = O.nms(boxes, scores, aidx, thr, n)
    rank = {i: r for r, i in enumerate(O.ranking(scores, aidx, n))}
    ks = set(kept)
    for i in kept:
        for j in kept:
            if i < j:
                assert O.iou(boxes[i], boxes[j]) <= thr
    for i in range(n):
        if i not in ks:  # suppressed by a kept box ranked before it
            assert any(rank[k] < rank[i] and O.iou(boxes[i], boxes[k]) > thr for k in kept)
    assert [int(aidx[i]) for i in kept] == sorted(int(aidx[i]) for i in kept)
