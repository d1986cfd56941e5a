"""fp64 oracle of rotated non-maximum suppression on bird's-eye-view boxes.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper's primary latency endpoint T^det ends when the final detections
exist: after box decoding, score thresholding and rotated NMS (Sec. V-A3).
The paper does not spell the NMS out; the readings used here:
  * the footprint of a box (x, y, z, w, l, h, yaw) is the rectangle centred
    at (x, y) whose side l lies along (cos yaw, sin yaw) and side w along
    (-sin yaw, cos yaw); overlap is the BEV intersection-over-union;
  * candidates are ranked by score, descending, ties by ascending anchor
    index, and only the first ``max_candidates`` take part;
  * greedy suppression: walking the ranking, a candidate is kept iff its IoU
    with every box kept before it is <= the threshold;
  * a box with a non-finite x, y, w, l or yaw, or with w <= 0 or l <= 0,
    overlaps nothing (IoU 0 with every box);
  * the kept boxes are reported in ascending anchor index.

The intersection area is computed from its plain definition: the footprint
of one box is intersected with the four half-planes bounded by the edges of
the other (textbook polygon clipping, one half-plane at a time; every
crossing point is computed once, so the clipped polygon is always closed),
and the shoelace formula gives the area of the result.
"""

import math

import numpy as np


def corners(box):
    """Footprint corners of one box, counter-clockwise, float64."""
    x, y, w, l, yaw = (float(box[0]), float(box[1]), float(box[3]), float(box[4]), float(box[6]))
    c, s = math.cos(yaw), math.sin(yaw)
    out = []
    for a, b in ((0.5, 0.5), (-0.5, 0.5), (-0.5, -0.5), (0.5, -0.5)):
        # a along the heading (length l), b across it (width w)
        out.append((x + a * l * c - b * w * s, y + a * l * s + b * w * c))
    return out


def valid(box):
    x, y, w, l, yaw = (float(box[0]), float(box[1]), float(box[3]), float(box[4]), float(box[6]))
    return all(math.isfinite(v) for v in (x, y, w, l, yaw)) and w > 0.0 and l > 0.0


def _cross(o, a, b):
    return (a[0] - o[0]) * (b[1] - o[1]) - (a[1] - o[1]) * (b[0] - o[0])


def clip_halfplane(poly, e0, e1):
    """Part of the polygon on the left of (or on) the directed line e0 -> e1."""
    out = []
    n = len(poly)
    for i in range(n):
        p, q = poly[i], poly[(i + 1) % n]
        fp, fq = _cross(e0, e1, p), _cross(e0, e1, q)
        if fp >= 0.0:
            out.append(p)
        if (fp >= 0.0) != (fq >= 0.0):
            t = fp / (fp - fq)
            out.append((p[0] + t * (q[0] - p[0]), p[1] + t * (q[1] - p[1])))
    return out


def polygon_area(pts):
    """Shoelace area of a simple polygon given in order."""
    n = len(pts)
    if n < 3:
        return 0.0
    s = 0.0
    for i in range(n):
        s += pts[i][0] * pts[(i + 1) % n][1] - pts[(i + 1) % n][0] * pts[i][1]
    return abs(s) * 0.5


def intersection_area(A, B):
    """Area of the intersection of two convex counter-clockwise polygons."""
    poly = list(A)
    for j in range(len(B)):
        poly = clip_halfplane(poly, B[j], B[(j + 1) % len(B)])
        if len(poly) < 3:
            return 0.0
    return polygon_area(poly)


def iou(a, b):
    """BEV intersection-over-union of two boxes (x, y, z, w, l, h, yaw)."""
    if not (valid(a) and valid(b)):
        return 0.0
    inter = intersection_area(corners(a), corners(b))
    union = float(a[3]) * float(a[4]) + float(b[3]) * float(b[4]) - inter
    return inter / union if union > 0.0 else 0.0


def _may_touch(a, others):
    """Exact pre-filter: footprints whose centres are farther apart than the
    sum of their circumradii cannot intersect (IoU 0)."""
    ra = 0.5 * math.hypot(float(a[3]), float(a[4]))
    rb = 0.5 * np.hypot(others[:, 3], others[:, 4])
    d = np.hypot(others[:, 0] - float(a[0]), others[:, 1] - float(a[1]))
    return ~(d > ra + rb)


def ranking(scores, anchor_idx, max_candidates):
    """Candidate order: score descending, ties by ascending anchor index."""
    order = sorted(range(len(scores)), key=lambda i: (-float(scores[i]), int(anchor_idx[i])))
    return order[:max_candidates]


def nms(boxes, scores, anchor_idx, iou_threshold, max_candidates):
    """Greedy rotated NMS; returns the indices (into the inputs) of the kept
    boxes in ascending anchor index."""
    boxes = np.asarray(boxes, dtype=np.float64).reshape(-1, 7)
    kept = []
    for i in ranking(scores, anchor_idx, max_candidates):
        if not valid(boxes[i]):
            kept.append(i)  # overlaps nothing, so nothing can suppress it
            continue
        if kept:
            kb = boxes[kept]
            near = [kept[j] for j in np.nonzero(_may_touch(boxes[i], kb))[0]]
        else:
            near = []
        if all(iou(boxes[i], boxes[k]) <= iou_threshold for k in near):
            kept.append(i)
    return sorted(kept, key=lambda i: int(anchor_idx[i]))
