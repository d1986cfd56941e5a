"""Shared helpers of the test suite: running frames through the C ABI and
comparing against the oracle."""

import time

import numpy as np

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
