"""Shared helpers of the test suite: running frames through the C ABI and
comparing against the oracle."""

import time

import numpy as np

from oracle import nms as ONMS
from paper_2608_08330_amd import rtcc as R

# Tolerances of the parity bar: max-norm relative error ||x - r||_inf / ||r||_inf
# against the fp64 oracle.
TOL = {"fp32": 1e-4, "bf16": 2e-2}


def rel_err(x, r):
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    den = np.max(np.abs(r)) if r.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(x))) if x.size else 0.0
    return float(np.max(np.abs(x - r)) / den)


def as_f32(raw, cfg):
    """Stored activation bytes -> float32 (bf16 bit patterns are widened)."""
    if cfg["precision"] == "bf16":
        return R.bf16_bits_to_f32(raw.view(np.uint16))
    return raw.view(np.float32)


def make_ctx(cfg, frame, max_points=None, **opt):
    o = R.rtcc_runtime_opts()
    o.exec = opt.get("exec", R.RTCC_EXEC_PER_BRANCH_STREAMS)
    o.use_graphs = opt.get("use_graphs", 0)
    o.node_timing = opt.get("node_timing", 0)
    o.device = 0
    o.premature_tol_s = opt.get("tol", 1e-6)
    n_max = max_points if max_points is not None else max(len(p) for p in frame["points"])
    return R.rtcc_create(R.model_desc(cfg, max(n_max, 1)), R.weights_blob(cfg, frame["weights"]), o,
                         kind=opt.get("kind", "gpu"))


def run_frame(ctx, frame, mode=R.RTCC_MODE_RELEASE, arrivals_s=None, points=None, realtime=False):
    """One frame: release branches in (a_k, k) order, join, detect.

    With ``realtime`` the call for agent k waits until t0 + a_k; otherwise
    t0 is placed far enough in the past that every event is on time."""
    cfg_points = frame["points"] if points is None else points
    K = len(cfg_points)
    a = np.zeros(K) if arrivals_s is None else np.asarray(arrivals_s, dtype=np.float64)
    R.rtcc_set_mode(ctx, mode)
    t0 = time.monotonic() - (0.0 if realtime else float(a.max()) + 1.0)
    R.rtcc_begin_frame(ctx, t0)
    for k in sorted(range(K), key=lambda k: (a[k], k)):
        if realtime:
            while time.monotonic() - t0 < a[k]:
                pass
        R.rtcc_release_branch(ctx, k, cfg_points[k], frame["poses"][k], float(a[k]))
    return R.rtcc_join_and_detect(ctx)


def tensors(ctx, cfg, with_stages=True):
    """Every tensor of the last frame as numpy (float32 for activations)."""
    K = cfg["K"]
    out = dict(cells=[], counts=[], canvas=[], slot=[], stage=[])
    for k in range(K):
        out["cells"].append(R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_CELLS, k, np.int32))
        out["counts"].append(R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_COUNTS, k, np.int32))
        out["canvas"].append(as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_CANVAS, k), cfg))
        out["slot"].append(as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_SLOT, k), cfg))
        if with_stages:
            out["stage"].append([as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_STAGE_OUT, (s << 8) | k), cfg)
                                 for s in range(len(cfg["stages"]))])
    out["fused"] = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg)
    out["head"] = R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32)
    return out


def compare_detections(det, ref, cfg, head_ref):
    """GPU detections vs the oracle's.

    Anchors whose oracle logit lies within tol * ||Z||_inf of the threshold
    may go either way; every other anchor must be kept by both or neither,
    and common boxes must agree to the precision's tolerance."""
    tol = TOL[cfg["precision"]]
    thr = cfg["logit_threshold"]
    logits = ref["logits"]
    band = tol * np.max(np.abs(head_ref))
    ambiguous = set(np.nonzero(np.abs(logits - thr) <= band)[0].tolist())
    g = set(det["anchor_idx"].tolist())
    o = set(ref["anchor_idx"].tolist())
    assert (g ^ o) <= ambiguous, sorted((g ^ o) - ambiguous)[:10]
    assert list(det["anchor_idx"]) == sorted(det["anchor_idx"])
    common = sorted(g & o)
    gi = {a: i for i, a in enumerate(det["anchor_idx"].tolist())}
    oi = {a: i for i, a in enumerate(ref["anchor_idx"].tolist())}
    if common:
        gb = det["boxes"][[gi[a] for a in common]]
        ob = ref["boxes"][[oi[a] for a in common]]
        # boxes: centres are O(10) m, sizes O(1); compare per column scale
        for col in range(7):
            scale = max(1.0, float(np.max(np.abs(ob[:, col]))))
            assert np.max(np.abs(gb[:, col] - ob[:, col])) <= 5 * tol * scale, col
        gs = det["scores"][[gi[a] for a in common]]
        os_ = ref["scores"][[oi[a] for a in common]]
        assert np.max(np.abs(gs - os_)) <= 5 * tol
    return len(common), len(ambiguous)


def nms_threshold(cfg):
    """The IoU threshold as the library stores it (float32), in float64."""
    return float(np.float32(cfg["nms_iou_threshold"]))


def ambiguous_pairs(boxes, thr, eps=1e-9):
    """Candidate pairs whose oracle IoU lies within eps of the threshold:
    float64 rounding of two different IoU algorithms may decide these
    either way."""
    b = np.asarray(boxes, dtype=np.float64)
    out = []
    for i in range(len(b)):
        for j in np.nonzero(ONMS._may_touch(b[i], b[i + 1:]))[0] + i + 1:
            if abs(ONMS.iou(b[i], b[j]) - thr) < eps:
                out.append((i, int(j)))
    return out


def check_nms(kept_idx, boxes, scores, anchor_idx, thr, max_candidates):
    """GPU NMS result (indices into the candidate records) against the
    oracle on the same float32 records: identical kept set; if the two
    differ, only pairs within rounding of the threshold may explain it and
    the GPU result must still be a valid greedy suppression."""
    b64 = np.asarray(boxes, dtype=np.float64)
    want = ONMS.nms(b64, scores, anchor_idx, thr, max_candidates)
    if list(kept_idx) == list(want):
        return len(want)
    amb = ambiguous_pairs(b64, thr)
    assert amb, ("NMS differs from the oracle", sorted(set(kept_idx) ^ set(want))[:10])
    order = ONMS.ranking(scores, anchor_idx, max_candidates)
    rank = {i: r for r, i in enumerate(order)}
    kept = set(kept_idx)
    assert kept <= set(order)
    for i in kept:
        for j in kept:
            if i < j:
                assert ONMS.iou(b64[i], b64[j]) <= thr + 1e-9
    for i in order:
        if i not in kept:
            assert any(rank[k] < rank[i] and ONMS.iou(b64[i], b64[k]) > thr - 1e-9 for k in kept)
    return len(kept)


def check_frame_nms(ctx, det, cfg):
    """The detections of the last frame are the oracle's NMS of the GPU's
    own decoded records (bit-identical records, identical kept set).
    Returns the decoded records for the decode-stage comparison."""
    dec = R.decoded_records(ctx)
    assert det["count_decoded"] == len(dec["anchor_idx"])
    assert list(dec["anchor_idx"]) == sorted(dec["anchor_idx"])
    pos = {int(a): i for i, a in enumerate(dec["anchor_idx"])}
    kept = [pos[int(a)] for a in det["anchor_idx"]]
    check_nms(kept, dec["boxes"], dec["scores"], dec["anchor_idx"], nms_threshold(cfg), cfg["nms_max_candidates"])
    assert np.array_equal(det["boxes"].view(np.uint32), dec["boxes"][kept].view(np.uint32))
    assert np.array_equal(det["scores"].view(np.uint32), dec["scores"][kept].view(np.uint32))
    return dec
