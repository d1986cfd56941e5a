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
    x = np.asarray(x, dtype=np.float64).ravel()
    r = np.asarray(r, dtype=np.float64).ravel()
    assert x.shape == r.shape, (x.shape, r.shape)
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
    o.conv_variant = opt.get("conv_variant", 0)
    o.conv_splits = opt.get("conv_splits", 0)
    if opt.get("torch_memory"):
        R.use_torch_memory(o, 0, opt.get("join_stream"))
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


# --------------------------------------------------------------- tight checks
# Checks of one kernel at a time: the oracle op applied to the GPU's own
# input of that op, so the only differences left are the summation order of
# float32 accumulation against float64 and, at a bf16 storage point, the
# rounding those differences can flip (one bf16 step, 2^-7 relative).  A
# tile-edge, halo or indexing error is far outside these bounds.

BF16_STEP = 2.0 ** -7


def tight(cfg):
    """(relative, floor) bounds of the one-kernel checks: one bf16 step at a
    bf16 storage point; float32 accumulation against float64 otherwise."""
    return (BF16_STEP, 1e-4) if cfg["precision"] == "bf16" else (1e-5, 1e-5)


def assert_close_elementwise(got, ref, rel, floor, what):
    """|got - ref| <= rel * |ref| + floor * max|ref| for every element."""
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    assert g.shape == r.shape, (what, g.shape, r.shape)
    scale = float(np.max(np.abs(r))) if r.size else 0.0
    bound = rel * np.abs(r) + floor * scale
    bad = np.nonzero(np.abs(g - r) > bound)[0]
    assert bad.size == 0, (what, "elements outside the bound", int(bad.size), "of", int(r.size), "first",
                           int(bad[0]), float(g[bad[0]]), float(r[bad[0]]))
    return float(np.max(np.abs(g - r)) / scale) if scale else 0.0


def check_decode_exact(ctx, cfg):
    """The GPU's decoded records against the oracle's decode of the GPU's
    own head output: the same anchors (the logit > threshold decision on the
    same float32 value and the float32 threshold), boxes to float32
    rounding of the residual decode, scores likewise.  A row / column mix-up
    or a half-cell shift of the anchor centres moves a box by a cell."""
    from oracle import network as ON
    H2, W2 = ON.feature_grid(cfg)
    head = R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32).reshape(H2, W2, 16).astype(np.float64)
    thr = float(np.float32(cfg["logit_threshold"]))
    ref = ON.decode(head, cfg, threshold=thr)
    dec = R.decoded_records(ctx)
    assert np.array_equal(dec["anchor_idx"].astype(np.int64), ref["anchor_idx"]), "decoded anchor set"
    n = len(ref["anchor_idx"])
    if n:
        for col in range(7):
            scale = max(1.0, float(np.max(np.abs(ref["boxes"][:, col]))))
            err = np.max(np.abs(dec["boxes"][:, col].astype(np.float64) - ref["boxes"][:, col]))
            assert err <= 1e-6 * scale, ("box column", col, err, scale)
        assert np.max(np.abs(dec["scores"].astype(np.float64) - ref["scores"])) <= 1e-6
    return n


def check_members(ctx, cfg, points, agent):
    """The points each pillar fed to the point-feature net, bit-exact: the
    lowest max_pts original indices of every pillar, pillars in cell order."""
    from oracle import network as ON
    pil = ON.pillars(ON.cell_ids(points, cfg), cfg["max_pts"])
    want = np.concatenate(pil["used"]).astype(np.int32) if pil["used"] else np.zeros(0, np.int32)
    got = R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_MEMBERS, agent, np.int32)
    assert np.array_equal(got, want), ("pillar members, agent", agent, got.size, want.size)
    return got.size


def conv_layer_shapes(cfg):
    """(stage, layer in stage, stride, C_in, C_out) of every 3x3 conv."""
    out = []
    c_in = cfg["c_pfn"]
    for s, (stride, c_out, n) in enumerate(cfg["stages"]):
        for l in range(n):
            out.append((s, l, stride if l == 0 else 1, c_in if l == 0 else c_out, c_out))
        c_in = c_out
    return out


def check_conv_layers(ctx, cfg, pw, agent, rel=None, floor=None):
    """Every 3x3 conv layer of one agent against the oracle conv of the
    GPU's own input to it (the canvas, then the previous layer's output),
    elementwise; then every upsampling into the slot from the GPU's stage
    outputs.  Returns the largest relative deviation per layer."""
    from oracle import network as ON
    if rel is None:
        rel, floor = tight(cfg)
    H, W = ON.grid(cfg)
    x = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_CANVAS, agent), cfg).reshape(H, W, -1)
    errs = []
    stage_out = []
    shapes = conv_layer_shapes(cfg)
    for li, (s, l, stride, _ci, co) in enumerate(shapes):
        ref = ON._store(cfg, ON.conv3x3(x.astype(np.float64), pw["s%dc%d_w" % (s, l)], pw["s%dc%d_b" % (s, l)],
                                        stride))
        got = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_CONV_OUT, (li << 8) | agent), cfg).reshape(ref.shape)
        errs.append(assert_close_elementwise(got, ref, rel, floor, ("conv layer", li, "agent", agent)))
        x = got
        if li + 1 == len(shapes) or shapes[li + 1][0] != s:
            stage_out.append(got)
    if cfg["up_channels"] and not cfg.get("multiscale"):
        H2, W2 = ON.feature_grid(cfg)
        slot = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_SLOT, agent), cfg).reshape(H2, W2, -1)
        up = cfg["up_channels"]
        rel_u = 1
        for s, (stride, _c, _n) in enumerate(cfg["stages"]):
            if s > 0:
                rel_u *= stride
            ref = ON._store(cfg, ON.deconv(stage_out[s].astype(np.float64), pw["up%d_w" % s], pw["up%d_b" % s],
                                           rel_u, H2, W2))
            errs.append(assert_close_elementwise(slot[:, :, s * up:(s + 1) * up], ref, rel, floor,
                                                 ("upsample", s, "agent", agent)))
    return errs


def check_fusion_and_head(ctx, cfg, poses, pw, rel=None, floor=None):
    """The fused map against the oracle warp + fusion of the GPU's own slots,
    and the head against the oracle head of the GPU's own fused map, both
    elementwise."""
    from oracle import network as ON
    if rel is None:
        rel, floor = (BF16_STEP, 1e-3) if cfg["precision"] == "bf16" else (1e-5, 1e-5)
    H2, W2 = ON.feature_grid(cfg)
    slots = [as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_SLOT, k), cfg).reshape(H2, W2, -1).astype(np.float64)
             for k in range(cfg["K"])]
    warped = [ON.warp(slots[k], poses[k], cfg) for k in range(cfg["K"])]
    fused_ref = ON._store(cfg, ON.fuse_attn(warped) if cfg["fusion"] == "attn" else ON.fuse_max(warped))
    fused = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg).reshape(H2, W2, -1)
    e_f = assert_close_elementwise(fused, fused_ref, rel, floor, "fusion")
    head_ref = ON.head(fused.astype(np.float64), pw["head_w"], pw["head_b"])
    head = R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32).reshape(H2, W2, 16)
    e_h = assert_close_elementwise(head, head_ref, 1e-5, 1e-5, "head")
    return e_f, e_h
