"""fp64 oracle of the fork-join intermediate-fusion detector.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper's DNN is a PointPillars-based intermediate-fusion detector: one
shared encoder instance per agent (Sec. V-A1), whose features are stored in
agent-indexed slots (Sec. IV-D) and, once all K encoders have finished,
fused and passed to the detection heads (Sec. III-B).  The paper does not
print the network's internals; the synthetic network here is the one of the
workload descriptions in ``synth/configs.py``; where the paper leaves a
point open, the reading taken is stated at the function that applies it.

Arithmetic is float64 except where a step is defined in lower precision:
  * the pillar cell index is computed in float32 (IEEE round-to-nearest
    subtract, divide, floor), so that both sides take the same integer
    decision in the same precision;
  * for bf16 workloads, weight matrices are rounded to bfloat16 and the
    activations are rounded to bfloat16 at the storage points of the network
    (canvas, every convolution / deconvolution output, fused map).

Every function is written from its definition: loops over taps or phases
with a matmul per tap as the only library primitive.
"""

import math

import numpy as np

from .bf16 import round_bf16


# ----------------------------------------------------------------------------
# geometry
# ----------------------------------------------------------------------------

def grid(cfg):
    """Pillar grid (H rows along y, W columns along x)."""
    W = int(round((cfg["x_range"][1] - cfg["x_range"][0]) / cfg["pillar"]))
    H = int(round((cfg["y_range"][1] - cfg["y_range"][0]) / cfg["pillar"]))
    return H, W


def stage_grids(cfg):
    """Output grid of every backbone stage: a 3x3, pad-1 convolution of
    stride s maps n cells to ceil(n / s)."""
    H, W = grid(cfg)
    out = []
    for stride, _c, _n in cfg["stages"]:
        H = -(-H // stride)
        W = -(-W // stride)
        out.append((H, W))
    return out


def feature_grid(cfg):
    """Grid of the agent slot / fused map / head: the first stage's output."""
    return stage_grids(cfg)[0]


def _is_bf16(cfg):
    return cfg["precision"] == "bf16"


def _store(cfg, x):
    """Storage-point rounding of an activation tensor."""
    return round_bf16(x) if _is_bf16(cfg) else x


def prepared_weights(cfg, weights):
    """float64 weights as the network uses them: weight matrices rounded to
    bfloat16 for bf16 workloads, biases kept at float32 precision."""
    out = {}
    for name, arr in weights.items():
        a = np.asarray(arr, dtype=np.float64)
        if name.endswith("_w") and _is_bf16(cfg):
            a = round_bf16(a)
        out[name] = a
    return out


# ----------------------------------------------------------------------------
# O1, O2: pillarization
# ----------------------------------------------------------------------------

def cell_ids(points, cfg):
    """Pillar cell of every point, or -1.

    A point (x, y, z, r) is kept iff all four values are finite and
    xmin <= x < xmax, ymin <= y < ymax, zmin <= z < zmax (float32
    comparisons).  Its column is floor(fl32(fl32(x - xmin) / fl32(v))) and
    its row likewise from y; a point whose index reaches W or H after
    rounding is dropped.  cell = row * W + col.
    """
    p = np.asarray(points, dtype=np.float32).reshape(-1, 4)
    H, W = grid(cfg)
    x0, x1 = (np.float32(v) for v in cfg["x_range"])
    y0, y1 = (np.float32(v) for v in cfg["y_range"])
    z0, z1 = (np.float32(v) for v in cfg["z_range"])
    v = np.float32(cfg["pillar"])
    x, y, z = p[:, 0], p[:, 1], p[:, 2]
    with np.errstate(invalid="ignore", over="ignore"):
        finite = np.isfinite(p).all(axis=1)
        inside = finite & (x >= x0) & (x < x1) & (y >= y0) & (y < y1) & (z >= z0) & (z < z1)
        fx = np.floor((x - x0) / v)
        fy = np.floor((y - y0) / v)
        ok = inside & (fx >= 0) & (fx < W) & (fy >= 0) & (fy < H)
    cell = np.full(p.shape[0], -1, dtype=np.int64)
    cell[ok] = fy[ok].astype(np.int64) * W + fx[ok].astype(np.int64)
    return cell


def pillars(cell, max_pts):
    """Group points by cell.

    Returns a dict with the non-empty cells in ascending order (``cells``),
    the number of points in each (``counts``), the point indices of each
    pillar in ascending original order (``members``, a list) and the points
    that enter the point-feature net, the lowest ``max_pts`` original
    indices of each pillar (``used``, a list).
    """
    cell = np.asarray(cell)
    valid = np.nonzero(cell >= 0)[0]
    order = np.argsort(cell[valid], kind="stable")
    sidx = valid[order]
    cells, start, counts = np.unique(cell[sidx], return_index=True, return_counts=True)
    members = [sidx[s:s + c] for s, c in zip(start, counts)]
    used = [m[:max_pts] for m in members]
    return dict(cells=cells.astype(np.int64), counts=counts.astype(np.int64),
                members=members, used=used)


# ----------------------------------------------------------------------------
# O3: point-feature net and dense canvas
# ----------------------------------------------------------------------------

def point_features(points, cfg):
    """(x / hx, y / hy, (z - zmin) / (zmax - zmin), r), hx and hy the half
    extents of the region: the raw point scaled to O(1)."""
    p = np.asarray(points, dtype=np.float64).reshape(-1, 4)
    hx = (cfg["x_range"][1] - cfg["x_range"][0]) / 2.0
    hy = (cfg["y_range"][1] - cfg["y_range"][0]) / 2.0
    dz = cfg["z_range"][1] - cfg["z_range"][0]
    f = np.empty_like(p)
    f[:, 0] = p[:, 0] / hx
    f[:, 1] = p[:, 1] / hy
    f[:, 2] = (p[:, 2] - cfg["z_range"][0]) / dz
    f[:, 3] = p[:, 3]
    return f


def pfn_canvas(points, pil, w, b, cfg):
    """Dense canvas [H, W, C]: for every pillar, the channel-wise max over
    its used points of ReLU(W^T f + b); empty cells are zero."""
    H, W = grid(cfg)
    C = w.shape[1]
    canvas = np.zeros((H * W, C), dtype=np.float64)
    if len(pil["cells"]):
        idx = np.concatenate(pil["used"])
        owner = np.repeat(pil["cells"], [len(u) for u in pil["used"]])
        f = point_features(np.asarray(points)[idx], cfg)
        h = np.maximum(f @ w + b, 0.0)
        # h >= 0 and each pillar has at least one point, so a zero start
        # value does not change the max.
        np.maximum.at(canvas, owner, h)
    return _store(cfg, canvas.reshape(H, W, C))


# ----------------------------------------------------------------------------
# O4, O5: backbone
# ----------------------------------------------------------------------------

def conv3x3(x, w, b, stride):
    """3x3 convolution, zero padding 1, given stride, bias, ReLU.

    out[y, x, o] = ReLU(b[o] + sum_{dy, dx in 0..2} sum_i
                        w[dy, dx, i, o] * in[s*y + dy - 1, s*x + dx - 1, i])
    with in = 0 outside the grid; the output has ceil(H / s) x ceil(W / s)
    cells.  Summed tap by tap, one matmul per tap.
    """
    H, W, Cin = x.shape
    Cout = w.shape[3]
    Ho, Wo = -(-H // stride), -(-W // stride)
    xp = np.zeros((H + 2, W + 2, Cin), dtype=np.float64)
    xp[1:-1, 1:-1] = x
    out = np.zeros((Ho, Wo, Cout), dtype=np.float64)
    for dy in range(3):
        for dx in range(3):
            patch = xp[dy:dy + stride * (Ho - 1) + 1:stride,
                       dx:dx + stride * (Wo - 1) + 1:stride]
            out += patch @ w[dy, dx]
    return np.maximum(out + b, 0.0)


def deconv(x, w, b, u, Ho, Wo):
    """Transposed convolution with kernel = stride = u, bias, ReLU, cropped
    to Ho x Wo:  out[y, x, c] = ReLU(b[c] + sum_i w[y mod u, x mod u, i, c]
    * in[y div u, x div u, i])."""
    Cout = w.shape[3]
    out = np.empty((Ho, Wo, Cout), dtype=np.float64)
    for py in range(u):
        for px in range(u):
            ys = np.arange(py, Ho, u)
            xs = np.arange(px, Wo, u)
            if len(ys) == 0 or len(xs) == 0:
                continue
            src = x[ys // u][:, xs // u]
            out[py::u, px::u] = src @ w[py, px] + b
    return np.maximum(out, 0.0)


def encoder(points, cfg, pw, keep=False):
    """One agent's encoder E_k: pillarize, point-feature net, backbone,
    upsample and concatenate.  Returns the slot tensor [H2, W2, C] and, if
    ``keep``, the intermediate tensors."""
    cell = cell_ids(points, cfg)
    pil = pillars(cell, cfg["max_pts"])
    canvas = pfn_canvas(points, pil, pw["pfn_w"], pw["pfn_b"], cfg)
    x = canvas
    stage_out = []
    for s, (stride, _c, n_convs) in enumerate(cfg["stages"]):
        for l in range(n_convs):
            x = _store(cfg, conv3x3(x, pw["s%dc%d_w" % (s, l)], pw["s%dc%d_b" % (s, l)],
                                    stride if l == 0 else 1))
        stage_out.append(x)
    if cfg["up_channels"]:
        H2, W2 = stage_out[0].shape[:2]
        parts = []
        rel = 1
        for s, (stride, _c, _n) in enumerate(cfg["stages"]):
            if s > 0:
                rel *= stride
            parts.append(_store(cfg, deconv(stage_out[s], pw["up%d_w" % s], pw["up%d_b" % s],
                                            rel, H2, W2)))
        slot = np.concatenate(parts, axis=2)
    else:
        slot = stage_out[-1]
    out = dict(slot=slot, cells=pil["cells"], counts=pil["counts"])
    if keep:
        out.update(cell=cell, pillars=pil, canvas=canvas, stage_out=stage_out)
    return out


# ----------------------------------------------------------------------------
# O7: pose warp
# ----------------------------------------------------------------------------

def cell_pitch(cfg, grid=None):
    """Cell size of a map of ``grid`` = (H, W) cells covering the BEV region
    (default: the feature grid)."""
    H2, W2 = feature_grid(cfg) if grid is None else grid
    dx = (cfg["x_range"][1] - cfg["x_range"][0]) / W2
    dy = (cfg["y_range"][1] - cfg["y_range"][0]) / H2
    return dx, dy


def sample_coords_metric(pose, cfg, grid=None):
    """Continuous agent-grid index (u = column, v = row) sampled by every
    ego cell, evaluated through metric coordinates.

    The ego cell (i, j) has centre p = (xmin + (j + 1/2) dx, ymin +
    (i + 1/2) dy).  The agent-to-ego pose maps agent points by
    p_ego = R(yaw) p_agent + t, so the ego cell pulls p_agent =
    R(yaw)^T (p - t), whose index on the agent's grid (cell centres at
    integer indices) is u = (p_agent.x - xmin) / dx - 1/2, likewise v.
    """
    H2, W2 = feature_grid(cfg) if grid is None else grid
    dx, dy = cell_pitch(cfg, grid)
    yaw, tx, ty = (float(v) for v in pose)
    c, s = math.cos(yaw), math.sin(yaw)
    jj, ii = np.meshgrid(np.arange(W2, dtype=np.float64), np.arange(H2, dtype=np.float64))
    px = cfg["x_range"][0] + (jj + 0.5) * dx - tx
    py = cfg["y_range"][0] + (ii + 0.5) * dy - ty
    ax = c * px + s * py
    ay = -s * px + c * py
    u = (ax - cfg["x_range"][0]) / dx - 0.5
    v = (ay - cfg["y_range"][0]) / dy - 0.5
    return u, v


def index_affine(pose, cfg, grid=None):
    """The same map written in index space: (u, v) = M (j, i) + t.

    With D = diag(dx, dy) and o the centre of cell (0, 0):
      M = D^-1 R^T D = [[c, s dy/dx], [-s dx/dy, c]]
      t = D^-1 (R^T (o - t_pose) - o)
    The identity pose gives M = I and t = 0 exactly.
    """
    dx, dy = cell_pitch(cfg, grid)
    yaw, tx, ty = (float(v) for v in pose)
    c, s = math.cos(yaw), math.sin(yaw)
    ox = cfg["x_range"][0] + 0.5 * dx
    oy = cfg["y_range"][0] + 0.5 * dy
    qx, qy = ox - tx, oy - ty
    rx = c * qx + s * qy
    ry = -s * qx + c * qy
    M = np.array([[c, s * dy / dx], [-s * dx / dy, c]], dtype=np.float64)
    t = np.array([(rx - ox) / dx, (ry - oy) / dy], dtype=np.float64)
    return M, t


def sample_coords(pose, cfg, grid=None):
    H2, W2 = feature_grid(cfg) if grid is None else grid
    M, t = index_affine(pose, cfg, grid)
    jj, ii = np.meshgrid(np.arange(W2, dtype=np.float64), np.arange(H2, dtype=np.float64))
    u = M[0, 0] * jj + M[0, 1] * ii + t[0]
    v = M[1, 0] * jj + M[1, 1] * ii + t[1]
    return u, v


def bilinear(X, u, v):
    """Bilinear sample of X [H, W, C] at continuous index (row v, column u);
    corners outside the grid contribute zero."""
    H, W, C = X.shape
    x0 = np.floor(u)
    y0 = np.floor(v)
    fx = u - x0
    fy = v - y0
    x0 = x0.astype(np.int64)
    y0 = y0.astype(np.int64)
    out = np.zeros(u.shape + (C,), dtype=np.float64)
    for oy, ox, wgt in ((0, 0, (1 - fx) * (1 - fy)), (0, 1, fx * (1 - fy)),
                        (1, 0, (1 - fx) * fy), (1, 1, fx * fy)):
        yy = y0 + oy
        xx = x0 + ox
        ok = (yy >= 0) & (yy < H) & (xx >= 0) & (xx < W)
        val = X[np.clip(yy, 0, H - 1), np.clip(xx, 0, W - 1)]
        out += np.where(ok, wgt, 0.0)[..., None] * val
    return out


def warp(slot, pose, cfg, grid=None):
    """Resample an agent's map [H, W, C] on the ego grid of the same size
    (``grid`` = (H, W); default the feature grid)."""
    u, v = sample_coords(pose, cfg, grid)
    return bilinear(slot, u, v)


# ----------------------------------------------------------------------------
# O8: fusion, O9: head, O10: decode
# ----------------------------------------------------------------------------

def fuse_max(warped):
    """Per cell, per channel maximum over the K agents."""
    return np.max(np.stack(warped, axis=0), axis=0)


def fuse_attn(warped):
    """Per-cell scaled dot-product attention across agents with the ego
    (agent 0) feature as the query and the K warped features as keys and
    values, no learned projections: s_k = <X_0, X_k> / sqrt(C),
    w = softmax(s), Y = sum_k w_k X_k."""
    X = np.stack(warped, axis=0)  # [K, H, W, C]
    C = X.shape[-1]
    s = np.einsum("hwc,khwc->khw", X[0], X) / math.sqrt(C)
    s = s - s.max(axis=0, keepdims=True)
    e = np.exp(s)
    wgt = e / e.sum(axis=0, keepdims=True)
    return np.einsum("khw,khwc->hwc", wgt, X)


def head(Y, w, b):
    """1x1 convolution C -> 2 anchors x (class logit + 7 box residuals)."""
    H, W, C = Y.shape
    return (Y.reshape(-1, C) @ w + b).reshape(H, W, -1)


def anchors(cfg):
    """Anchor boxes [H2, W2, A, 7] = (x, y, z, w, l, h, yaw): one per yaw at
    every feature-cell centre."""
    H2, W2 = feature_grid(cfg)
    dx, dy = cell_pitch(cfg)
    A = cfg["n_anchors"]
    out = np.zeros((H2, W2, A, 7), dtype=np.float64)
    jj, ii = np.meshgrid(np.arange(W2, dtype=np.float64), np.arange(H2, dtype=np.float64))
    for a in range(A):
        out[:, :, a, 0] = cfg["x_range"][0] + (jj + 0.5) * dx
        out[:, :, a, 1] = cfg["y_range"][0] + (ii + 0.5) * dy
        out[:, :, a, 2] = cfg["anchor_z"]
        out[:, :, a, 3] = cfg["anchor_w"]
        out[:, :, a, 4] = cfg["anchor_l"]
        out[:, :, a, 5] = cfg["anchor_h"]
        out[:, :, a, 6] = cfg["anchor_yaws"][a]
    return out


def decode(Z, cfg, threshold=None):
    """Threshold and decode the head output.

    An anchor is kept iff its class logit exceeds the threshold (strictly).
    Residual box coding: with d = sqrt(w_a^2 + l_a^2),
      x = x_a + dx d, y = y_a + dy d, z = z_a + dz h_a,
      w = w_a e^dw, l = l_a e^dl, h = h_a e^dh, yaw = yaw_a + dyaw,
    score = 1 / (1 + e^-logit).  Kept anchors are listed in ascending
    anchor index (row * W2 + col) * A + a.
    """
    tau = cfg["logit_threshold"] if threshold is None else threshold
    H2, W2 = Z.shape[:2]
    A = cfg["n_anchors"]
    Zr = Z.reshape(H2 * W2 * A, 8)
    anc = anchors(cfg).reshape(H2 * W2 * A, 7)
    keep = np.nonzero(Zr[:, 0] > tau)[0]
    r = Zr[keep]
    a = anc[keep]
    diag = np.sqrt(a[:, 3] ** 2 + a[:, 4] ** 2)
    boxes = np.empty((len(keep), 7), dtype=np.float64)
    boxes[:, 0] = a[:, 0] + r[:, 1] * diag
    boxes[:, 1] = a[:, 1] + r[:, 2] * diag
    boxes[:, 2] = a[:, 2] + r[:, 3] * a[:, 5]
    boxes[:, 3] = a[:, 3] * np.exp(r[:, 4])
    boxes[:, 4] = a[:, 4] * np.exp(r[:, 5])
    boxes[:, 5] = a[:, 5] * np.exp(r[:, 6])
    boxes[:, 6] = a[:, 6] + r[:, 7]
    scores = 1.0 / (1.0 + np.exp(-r[:, 0]))
    return dict(anchor_idx=keep.astype(np.int64), boxes=boxes, scores=scores,
                logits=Zr[:, 0])


# ----------------------------------------------------------------------------
# whole frame
# ----------------------------------------------------------------------------

def forward(frame, keep=False, agents=None):
    """Complete inference output of one frame.

    The result is a function of the inputs and weights only: it is the
    same for every arrival and release vector, which is the output
    invariance RTCC preserves (Sec. IV-D: fixed agent-indexed feature
    storage, post-join subgraph in topological order).

    With ``cfg['multiscale']`` the agents are fused at every backbone scale
    before upsampling (see :func:`_forward_multiscale`).

    With ``cfg['warp_in_branch']`` the pose warp moves out of the shared
    subgraph into each branch (a dependency-preserving move: the warp of
    agent k needs only E_k's slot and k's pose), which then stores its
    ego-frame map; the join fuses the K stored maps.
    """
    cfg = frame["cfg"]
    pw = prepared_weights(cfg, frame["weights"])
    K = cfg["K"]
    if cfg.get("multiscale"):
        return _forward_multiscale(frame, pw, keep)
    enc = [encoder(frame["points"][k], cfg, pw, keep=keep) for k in range(K)]
    warped = [warp(enc[k]["slot"], frame["poses"][k], cfg) for k in range(K)]
    if cfg.get("warp_in_branch"):
        # the warp is the last node of each branch, which stores its
        # ego-frame map: a storage point (rounded for bf16 workloads)
        warped = [_store(cfg, w) for w in warped]
    if cfg["fusion"] == "max":
        fused = fuse_max(warped)
    elif cfg["fusion"] == "attn":
        fused = fuse_attn(warped)
    else:
        raise ValueError(cfg["fusion"])
    fused = _store(cfg, fused)
    Z = head(fused, pw["head_w"], pw["head_b"])
    det = decode(Z, cfg)
    out = dict(enc=enc, fused=fused, head=Z, det=det)
    if keep:
        out["warped"] = warped
    return out


def _fuse(cfg, warped):
    if cfg["fusion"] == "max":
        return fuse_max(warped)
    if cfg["fusion"] == "attn":
        return fuse_attn(warped)
    raise ValueError(cfg["fusion"])


def _forward_multiscale(frame, pw, keep):
    """Multi-scale fusion: the branch E_k ends at its backbone stage outputs;
    the shared subgraph warps every agent's stage-s map onto the ego grid of
    stage s (H_s x W_s cells covering the BEV region, cell-centre
    convention), fuses the K maps of each scale, upsamples every fused map
    to the feature grid (transposed convolution, kernel = stride =
    2^s, bias, ReLU, crop), concatenates the scales and runs the head.
    Storage points (bf16 workloads): the fused map of each scale and each
    upsampled map."""
    cfg = frame["cfg"]
    K = cfg["K"]
    if not cfg["up_channels"]:
        raise ValueError("multi-scale fusion needs the upsampling stages")
    enc = [encoder(frame["points"][k], cfg, pw, keep=True) for k in range(K)]
    grids = stage_grids(cfg)
    H2, W2 = feature_grid(cfg)
    fused_s, parts, warped_s = [], [], []
    rel = 1
    for s, (stride, _c, _n) in enumerate(cfg["stages"]):
        if s > 0:
            rel *= stride
        warped = [warp(enc[k]["stage_out"][s], frame["poses"][k], cfg, grids[s]) for k in range(K)]
        f = _store(cfg, _fuse(cfg, warped))
        fused_s.append(f)
        parts.append(_store(cfg, deconv(f, pw["up%d_w" % s], pw["up%d_b" % s], rel, H2, W2)))
        if keep:
            warped_s.append(warped)
    fused = np.concatenate(parts, axis=2)
    Z = head(fused, pw["head_w"], pw["head_b"])
    det = decode(Z, cfg)
    out = dict(enc=enc, fused=fused, fused_stages=fused_s, head=Z, det=det)
    if keep:
        out["warped_stages"] = warped_s
    return out
