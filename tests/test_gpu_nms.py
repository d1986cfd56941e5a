"""GPU rotated NMS (rtcc_rotated_nms, the kernels that end the join) against
the oracle on the same float32 records: identical kept sets, including score
ties, identical and invalid boxes, the candidate cap and the largest cap."""

import math
import sys

import numpy as np
import pytest

from paper_2608_08330_amd import rtcc as R
from tests.helpers import check_nms

pytestmark = pytest.mark.gpu


def _records(boxes, scores, anchors):
    n = len(scores)
    rec = np.zeros((n, 9), dtype=np.float32)
    rec[:, :7] = boxes
    rec[:, 7] = scores
    rec[:, 8] = np.asarray(anchors, dtype=np.int32).view(np.float32)
    return rec


def _gpu_nms(rec, max_cand, thr):
    import torch
    n = len(rec)
    d_rec = torch.from_numpy(np.ascontiguousarray(rec)).to("cuda") if n else torch.zeros((1, 9), device="cuda")
    d_out = torch.zeros((max(1, min(n, max_cand)), 9), dtype=torch.float32, device="cuda")
    kept = R.rtcc_rotated_nms(d_rec.data_ptr(), n, max_cand, thr, d_out.data_ptr())
    torch.cuda.synchronize()
    return d_out[:kept].cpu().numpy()


def _scene(rng, n, spread, clusters=0):
    if clusters:
        c = rng.uniform(-spread, spread, (clusters, 2))
        xy = c[rng.integers(0, clusters, n)] + rng.normal(0, 1.0, (n, 2))
    else:
        xy = rng.uniform(-spread, spread, (n, 2))
    boxes = np.zeros((n, 7), dtype=np.float32)
    boxes[:, 0:2] = xy
    boxes[:, 2] = -1.0
    boxes[:, 3] = rng.uniform(1.2, 2.2, n)
    boxes[:, 4] = rng.uniform(3.0, 5.0, n)
    boxes[:, 5] = 1.5
    boxes[:, 6] = rng.uniform(-math.pi, math.pi, n)
    anchors = np.sort(rng.choice(10 * n + 10, n, replace=False)).astype(np.int32)
    return boxes, rng.uniform(0.3, 1.0, n).astype(np.float32), anchors


def _check(boxes, scores, anchors, max_cand, thr, label):
    print("nms case %s: n=%d cap=%d thr=%g" % (label, len(scores), max_cand, thr), flush=True)
    sys.stdout.flush()
    rec = _records(boxes, scores, anchors)
    out = _gpu_nms(rec, max_cand, thr)
    pos = {int(a): i for i, a in enumerate(anchors)}
    got_anchor = out[:, 8].copy().view(np.int32)
    assert list(got_anchor) == sorted(got_anchor)
    kept = [pos[int(a)] for a in got_anchor]
    assert np.array_equal(out.view(np.uint32), rec[kept].view(np.uint32))
    return check_nms(kept, boxes, scores, anchors, float(np.float32(thr)), max_cand)


@pytest.mark.parametrize("seed,n,spread,clusters,cap,thr", [
    (1, 1500, 60.0, 40, 4096, 0.15),   # clustered, below the cap
    (2, 3000, 40.0, 30, 1000, 0.15),   # more decoded boxes than candidates
    (3, 700, 15.0, 0, 4096, 0.0),      # any overlap suppresses
    (4, 700, 15.0, 0, 4096, 0.5),
    (5, 129, 5.0, 0, 64, 0.15),        # ragged: cap and count not multiples of 64
    (6, 4096, 6.0, 0, 4096, 0.15),     # dense: more listed mask words than the walk holds in LDS
])
def test_random_scenes(seed, n, spread, clusters, cap, thr):
    rng = np.random.default_rng(seed)
    boxes, scores, anchors = _scene(rng, n, spread, clusters)
    kept = _check(boxes, scores, anchors, cap, thr, "random %d" % seed)
    assert 0 < kept <= min(n, cap)


def test_ties_identical_and_invalid_boxes():
    rng = np.random.default_rng(9)
    boxes, scores, anchors = _scene(rng, 300, 10.0, 5)
    scores[:] = 0.75                   # every score tied: anchor order decides
    boxes[10] = boxes[11]              # identical pairs
    boxes[20] = boxes[21]
    boxes[30, 0] = np.nan              # invalid footprints overlap nothing
    boxes[31, 3] = np.inf
    boxes[32, 4] = 0.0
    boxes[33, 6] = np.nan
    kept = _check(boxes, scores, anchors, 4096, 0.15, "ties")
    assert kept > 0
    for thr in (1.0, 0.999):
        _check(boxes, scores, anchors, 4096, thr, "ties thr %g" % thr)


def test_single_and_empty():
    rng = np.random.default_rng(4)
    boxes, scores, anchors = _scene(rng, 1, 1.0)
    assert _check(boxes, scores, anchors, 1, 0.15, "single") == 1
    import torch
    d_out = torch.zeros((1, 9), dtype=torch.float32, device="cuda")
    assert R.rtcc_rotated_nms(0, 0, 16, 0.15, d_out.data_ptr()) == 0


def test_largest_candidate_cap():
    rng = np.random.default_rng(12)
    boxes, scores, anchors = _scene(rng, 20000, 400.0, 0)
    kept = _check(boxes, scores, anchors, 16384, 0.15, "cap 16384")
    assert 12000 < kept <= 16384


def test_argument_errors():
    import torch
    d = torch.zeros((4, 9), dtype=torch.float32, device="cuda")
    for args in ((d.data_ptr(), 4, 0, 0.15), (d.data_ptr(), 4, 16385, 0.15), (d.data_ptr(), 4, 16, 1.5),
                 (d.data_ptr(), 4, 16, -0.1), (d.data_ptr(), -1, 16, 0.15), (0, 4, 16, 0.15)):
        with pytest.raises(R.RtccError):
            R.rtcc_rotated_nms(args[0], args[1], args[2], args[3], d.data_ptr())


def test_shared_edges_and_nearly_parallel_edges():
    # footprints on an integer grid with yaw a multiple of pi/2 (edges that
    # coincide up to the rounding of cos / sin), and copies turned by 1e-9
    # to 1e-4 rad (nearly parallel edges)
    rng = np.random.default_rng(21)
    n = 600
    boxes = np.zeros((n, 7), dtype=np.float32)
    boxes[:, 0:2] = rng.integers(-6, 6, (n, 2))
    boxes[:, 3:5] = rng.integers(1, 4, (n, 2))
    boxes[:, 5] = 1.5
    boxes[:, 6] = (rng.integers(0, 4, n) * (math.pi / 2)).astype(np.float32)
    tilt = rng.random(n) < 0.3
    boxes[tilt, 6] += (10.0 ** rng.uniform(-9, -4, tilt.sum())).astype(np.float32)
    scores = rng.uniform(0.3, 1.0, n).astype(np.float32)
    anchors = np.arange(n, dtype=np.int32) * 3
    for thr in (0.15, 0.5):
        _check(boxes, scores, anchors, 4096, thr, "grid thr %g" % thr)


def test_negative_and_signed_zero_scores():
    """Scores of either sign (raw logits, say) rank by value: negative scores
    rank below positive ones and among themselves by magnitude, -0 ties +0
    (broken by anchor index), infinities at the ends."""
    rng = np.random.default_rng(31)
    boxes, _, anchors = _scene(rng, 800, 12.0, 6)
    scores = rng.normal(0.0, 3.0, 800).astype(np.float32)
    scores[:40] = -scores[40:80]           # mirrored pairs
    scores[100:110] = 0.0
    scores[110:120] = -0.0
    scores[200] = np.inf
    scores[201] = -np.inf
    for cap, thr in ((4096, 0.15), (300, 0.15), (4096, 0.0)):
        kept = _check(boxes, scores, anchors, cap, thr, "signed cap %d thr %g" % (cap, thr))
        assert kept > 0


def test_nan_score_rejected():
    rng = np.random.default_rng(32)
    boxes, scores, anchors = _scene(rng, 50, 5.0)
    scores[17] = np.nan
    rec = _records(boxes, scores, anchors)
    with pytest.raises(R.RtccError) as e:
        _gpu_nms(rec, 64, 0.15)
    assert e.value.status == R.RTCC_E_ARG
