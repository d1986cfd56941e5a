"""Pins of the oracle's point-feature net, convolution, deconvolution, pose
warp, fusion, head and decode: closed forms, direct summation, special
cases that reduce to numpy routines, and library cross-checks."""

import math

import numpy as np
import pytest

import synth
from oracle import network as N
from oracle.bf16 import round_bf16


# ---------------------------------------------------------------- PFN

def test_pfn_identity_weights_closed_form():
    cfg = synth.config("c1")
    H, W = N.grid(cfg)
    rng = np.random.default_rng(0)
    pts = np.zeros((40, 4), dtype=np.float32)
    pts[:, 0] = rng.uniform(-25.6, 25.6, 40)
    pts[:, 1] = rng.uniform(-25.6, 25.6, 40)
    pts[:, 2] = rng.uniform(-3, 1, 40)
    pts[:, 3] = rng.uniform(0, 1, 40)
    pts[:10, :2] = [1.0, 1.0]  # ten points in one pillar
    cell = N.cell_ids(pts, cfg)
    pil = N.pillars(cell, 32)
    canvas = N.pfn_canvas(pts, pil, np.eye(4), np.zeros(4), cfg)
    # closed form: per coordinate max of ReLU(feature) over the pillar
    for p, c in enumerate(pil["cells"]):
        m = pil["members"][p]
        f = np.stack([pts[m, 0] / 25.6, pts[m, 1] / 25.6, (pts[m, 2] + 3.0) / 4.0, pts[m, 3]], 1)
        np.testing.assert_allclose(canvas.reshape(-1, 4)[c], np.maximum(f, 0).max(0), rtol=1e-6)
    empty = np.setdiff1d(np.arange(H * W), pil["cells"])
    assert np.all(canvas.reshape(-1, 4)[empty] == 0)


def test_pfn_single_point_pillar():
    cfg = synth.config("c1")
    pts = np.array([[12.8, -6.4, -1.0, 0.25]], dtype=np.float32)
    pil = N.pillars(N.cell_ids(pts, cfg), 32)
    w = np.array([[1.0, -1.0], [2.0, 0.0], [0.0, 4.0], [1.0, 1.0]])
    b = np.array([0.1, -3.0])
    canvas = N.pfn_canvas(pts, pil, w, b, cfg)
    # features by hand: 12.8/25.6 = 0.5, -6.4/25.6 = -0.25, (-1+3)/4 = 0.5, 0.25
    f = np.array([0.5, -0.25, 0.5, 0.25])
    want = np.maximum(f @ w + b, 0)  # [0.1 + 0.5 - 0.5 + 0.25, ...] = [0.35, 0]
    np.testing.assert_allclose(want, [0.35, 0.0], atol=1e-6)
    np.testing.assert_allclose(canvas.reshape(-1, 2)[pil["cells"][0]], want, rtol=1e-6, atol=1e-7)


# ---------------------------------------------------------------- conv

def _direct_conv(x, w, b, s):
    H, W, Ci = x.shape
    Co = w.shape[3]
    Ho, Wo = -(-H // s), -(-W // s)
    out = np.zeros((Ho, Wo, Co))
    for y in range(Ho):
        for xx in range(Wo):
            for o in range(Co):
                acc = b[o]
                for dy in range(3):
                    for dx in range(3):
                        iy, ix = s * y + dy - 1, s * xx + dx - 1
                        if 0 <= iy < H and 0 <= ix < W:
                            for i in range(Ci):
                                acc += w[dy, dx, i, o] * x[iy, ix, i]
                out[y, xx, o] = max(acc, 0.0)
    return out


@pytest.mark.parametrize("shape,stride", [((5, 6, 3), 1), ((5, 6, 3), 2), ((7, 5, 2), 2)])
def test_conv_direct_summation(shape, stride):
    rng = np.random.default_rng(11)
    x = rng.standard_normal(shape)
    w = rng.standard_normal((3, 3, shape[2], 4))
    b = rng.standard_normal(4)
    np.testing.assert_allclose(N.conv3x3(x, w, b, stride), _direct_conv(x, w, b, stride),
                               rtol=1e-12, atol=1e-12)


def test_conv_delta_kernel_shifts_and_identity():
    rng = np.random.default_rng(2)
    x = np.abs(rng.standard_normal((6, 7, 3)))
    w = np.zeros((3, 3, 3, 3))
    for i in range(3):
        w[1, 1, i, i] = 1.0
    assert np.array_equal(N.conv3x3(x, w, np.zeros(3), 1), x)
    w = np.zeros((3, 3, 3, 3))
    for i in range(3):
        w[0, 2, i, i] = 1.0  # reads in[y - 1, x + 1]
    out = N.conv3x3(x, w, np.zeros(3), 1)
    want = np.zeros_like(x)
    want[1:, :-1] = x[:-1, 1:]
    assert np.array_equal(out, want)


# ---------------------------------------------------------------- deconv

def test_deconv_u1_is_pointwise_matmul():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((5, 7, 6))
    w = rng.standard_normal((1, 1, 6, 3))
    b = rng.standard_normal(3)
    ref = np.maximum(np.matmul(x.reshape(-1, 6), w[0, 0]).reshape(5, 7, 3) + b, 0)
    np.testing.assert_allclose(N.deconv(x, w, b, 1, 5, 7), ref, rtol=1e-13, atol=1e-13)


def test_deconv_one_hot_is_nearest_upsample_with_crop():
    rng = np.random.default_rng(5)
    x = np.abs(rng.standard_normal((3, 4, 2)))
    u = 4
    w = np.zeros((u, u, 2, 2))
    for py in range(u):
        for px in range(u):
            w[py, px] = np.eye(2)
    up = np.repeat(np.repeat(x, u, axis=0), u, axis=1)
    assert np.array_equal(N.deconv(x, w, np.zeros(2), u, 10, 15), up[:10, :15])


def test_deconv_phase_weights():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 2, 1))
    w = rng.standard_normal((2, 2, 1, 1))
    out = N.deconv(x, w, np.zeros(1), 2, 4, 4)
    for y in range(4):
        for xx in range(4):
            assert out[y, xx, 0] == max(w[y % 2, xx % 2, 0, 0] * x[y // 2, xx // 2, 0], 0.0)


# ---------------------------------------------------------------- warp

def test_identity_pose_is_exact_identity():
    for name in ("c1", "t_max", "c3"):
        cfg = synth.config(name)
        H2, W2 = N.feature_grid(cfg)
        M, t = N.index_affine((0.0, 0.0, 0.0), cfg)
        assert np.array_equal(M, np.eye(2)) and np.array_equal(t, np.zeros(2))
        X = np.random.default_rng(0).standard_normal((H2, W2, 5))
        assert np.array_equal(N.warp(X, (0.0, 0.0, 0.0), cfg), X)


def test_index_affine_matches_metric_definition():
    rng = np.random.default_rng(9)
    for name in ("c1", "c3", "t_attn"):
        cfg = synth.config(name)
        for _ in range(5):
            pose = (rng.uniform(-math.pi, math.pi), rng.uniform(-5, 5), rng.uniform(-5, 5))
            u1, v1 = N.sample_coords(pose, cfg)
            u2, v2 = N.sample_coords_metric(pose, cfg)
            np.testing.assert_allclose(u1, u2, atol=1e-9)
            np.testing.assert_allclose(v1, v2, atol=1e-9)


def test_whole_cell_translation_shifts_with_zero_fill():
    cfg = synth.config("c1")  # feature cell pitch 0.8 m
    H2, W2 = N.feature_grid(cfg)
    X = np.random.default_rng(1).standard_normal((H2, W2, 3))
    # agent frame is ego frame shifted by t = (2 cells in x, -1 cell in y):
    # ego cell (i, j) pulls agent cell (i + 1, j - 2)
    Y = N.warp(X, (0.0, 1.6, -0.8), cfg)
    want = np.zeros_like(X)
    want[:-1, 2:] = X[1:, :-2]
    np.testing.assert_allclose(Y, want, atol=1e-12)


def test_quarter_turn_is_rot90():
    cfg = synth.config("c1")  # square, symmetric grid
    H2, W2 = N.feature_grid(cfg)
    X = np.random.default_rng(2).standard_normal((H2, W2, 2))
    Y = N.warp(X, (math.pi / 2, 0.0, 0.0), cfg)
    np.testing.assert_allclose(Y, np.rot90(X, k=-1, axes=(0, 1)), atol=1e-9)


def test_half_cell_shift_is_neighbour_mean():
    cfg = synth.config("c1")
    H2, W2 = N.feature_grid(cfg)
    X = np.random.default_rng(3).standard_normal((H2, W2, 2))
    Y = N.warp(X, (0.0, -0.4, 0.0), cfg)  # ego (i, j) pulls agent column j + 1/2
    np.testing.assert_allclose(Y[:, :-1], 0.5 * (X[:, :-1] + X[:, 1:]), atol=1e-12)
    np.testing.assert_allclose(Y[:, -1], 0.5 * X[:, -1], atol=1e-12)


# ---------------------------------------------------------------- fusion

def test_single_agent_fusion_is_identity():
    X = np.abs(np.random.default_rng(0).standard_normal((4, 5, 8)))
    assert np.array_equal(N.fuse_max([X]), X)
    assert np.array_equal(N.fuse_attn([X]), X)


def test_identical_agents_attention_returns_features():
    X = np.abs(np.random.default_rng(1).standard_normal((4, 5, 8)))
    np.testing.assert_allclose(N.fuse_attn([X, X, X]), X, rtol=1e-14)
    Y = np.maximum(X - 0.3, 0)
    assert np.array_equal(N.fuse_max([X, Y]), X)


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    K, H, W, C = 4, 3, 5, 16
    Xs = [np.abs(rng.standard_normal((H, W, C))) for _ in range(K)]
    got = N.fuse_attn(Xs)
    X = torch.from_numpy(np.stack(Xs, 0)).permute(1, 2, 0, 3).reshape(H * W, K, C)
    ref = torch.nn.functional.scaled_dot_product_attention(X, X, X)  # [HW, K, C]
    np.testing.assert_allclose(got, ref[:, 0, :].reshape(H, W, C).numpy(), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- head, decode

def test_head_matches_explicit_sum():
    rng = np.random.default_rng(3)
    Y = rng.standard_normal((3, 4, 6))
    w = rng.standard_normal((6, 16))
    b = rng.standard_normal(16)
    Z = N.head(Y, w, b)
    for i in range(3):
        for j in range(4):
            for o in range(16):
                assert abs(Z[i, j, o] - (b[o] + sum(Y[i, j, c] * w[c, o] for c in range(6)))) < 1e-12


def test_decode_zero_residuals_give_anchors():
    cfg = synth.config("c1")
    H2, W2 = N.feature_grid(cfg)
    Z = np.zeros((H2, W2, 16))
    Z[..., 0] = 5.0
    Z[..., 8] = 5.0
    det = N.decode(Z, cfg)
    assert len(det["anchor_idx"]) == H2 * W2 * 2
    np.testing.assert_array_equal(det["boxes"], N.anchors(cfg).reshape(-1, 7))
    np.testing.assert_allclose(det["scores"], 1 / (1 + math.exp(-5.0)))
    # anchor (0, 0, 0) centre is the first cell centre
    assert det["boxes"][0, 0] == -25.6 + 0.4 and det["boxes"][0, 1] == -25.6 + 0.4


def test_decode_single_anchor_by_hand_and_strict_threshold():
    cfg = synth.config("c1")
    H2, W2 = N.feature_grid(cfg)
    tau = cfg["logit_threshold"]
    Z = np.full((H2, W2, 16), -10.0)
    i, j = 10, 20
    Z[i, j, 8:16] = [2.0, 0.1, -0.2, 0.5, math.log(2.0), 0.0, math.log(0.5), 0.3]
    Z[3, 4, 0] = tau  # equal to the threshold: dropped
    det = N.decode(Z, cfg)
    assert det["anchor_idx"].tolist() == [(i * W2 + j) * 2 + 1]
    d = math.sqrt(1.6 ** 2 + 3.9 ** 2)
    xa = -25.6 + (j + 0.5) * 0.8
    ya = -25.6 + (i + 0.5) * 0.8
    want = [xa + 0.1 * d, ya - 0.2 * d, -1.0 + 0.5 * 1.5, 3.2, 3.9, 0.75, math.pi / 2 + 0.3]
    np.testing.assert_allclose(det["boxes"][0], want, rtol=1e-12)
    np.testing.assert_allclose(det["scores"][0], 1 / (1 + math.exp(-2.0)))


def test_forward_output_does_not_depend_on_agent_slot_order():
    """Fixed-index storage: fusion reads slots by agent index, so computing
    the encoders in any order gives the same frame output."""
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    out = N.forward(fr)
    pw = N.prepared_weights(cfg, fr["weights"])
    rev = {k: N.encoder(fr["points"][k], cfg, pw)["slot"] for k in reversed(range(cfg["K"]))}
    warped = [N.warp(rev[k], fr["poses"][k], cfg) for k in range(cfg["K"])]
    fused = N._store(cfg, N.fuse_attn(warped))
    assert np.array_equal(fused, out["fused"])


def _prewarp(cfg, on=True):
    c = dict(cfg)
    c["warp_in_branch"] = on
    return c


@pytest.mark.parametrize("name", ["t_max", "c1"])
def test_prewarp_max_fusion_equals_post_join_warp(name):
    """Rounding to bfloat16 is monotone, so the maximum of the rounded
    ego-frame maps is the rounded maximum: with max fusion, storing each
    branch's warped map changes nothing (c1 is float32: no rounding)."""
    fr = synth.make_frame(name)
    base = N.forward(fr)
    fr2 = dict(fr, cfg=_prewarp(fr["cfg"]))
    pre = N.forward(fr2, keep=True)
    assert np.array_equal(pre["fused"], base["fused"])
    assert np.array_equal(pre["head"], base["head"])
    if fr["cfg"]["precision"] == "bf16":
        for w in pre["warped"]:
            assert np.array_equal(w, round_bf16(w))


def test_prewarp_attention_identity_poses_and_single_agent():
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    # identity poses: every warp is the identity on bf16 slots, so the stored
    # maps equal the slots and both placements fuse the same values
    ident = dict(fr, poses=np.zeros_like(fr["poses"]))
    a = N.forward(ident)
    b = N.forward(dict(ident, cfg=_prewarp(cfg)))
    assert np.array_equal(a["fused"], b["fused"])
    # one agent: attention returns its (stored) warped map
    one = dict(cfg, K=1, warp_in_branch=True)
    fr1 = dict(fr, cfg=one, points=fr["points"][:1], poses=fr["poses"][:1])
    out = N.forward(fr1, keep=True)
    assert np.array_equal(out["fused"], N._store(one, out["warped"][0]))
    # random poses: the two placements differ only by the rounding of the
    # warped maps (relative 2^-8 per element before fusion)
    c = N.forward(fr)
    d = N.forward(dict(fr, cfg=_prewarp(cfg)))
    scale = np.abs(c["fused"]).max()
    assert np.abs(c["fused"] - d["fused"]).max() <= 2 ** -7 * scale
    assert not np.array_equal(c["fused"], d["fused"])


def _multiscale(cfg):
    c = dict(cfg)
    c["multiscale"] = True
    return c


def test_stage_grid_warp_identity_and_metric_consistency():
    cfg = synth.config("c3")  # ragged stage grids: 50 x 176, 25 x 88, 13 x 44
    for g in N.stage_grids(cfg):
        M, t = N.index_affine((0.0, 0.0, 0.0), cfg, g)
        assert np.array_equal(M, np.eye(2)) and np.array_equal(t, np.zeros(2))
        pose = (0.7, 2.3, -1.9)
        u1, v1 = N.sample_coords(pose, cfg, g)
        u2, v2 = N.sample_coords_metric(pose, cfg, g)
        np.testing.assert_allclose(u1, u2, atol=1e-9)
        np.testing.assert_allclose(v1, v2, atol=1e-9)


def test_stage_grid_whole_cell_translation():
    cfg = synth.config("t_attn")
    g = N.stage_grids(cfg)[1]
    dx, dy = N.cell_pitch(cfg, g)
    rng = np.random.default_rng(2)
    X = rng.uniform(0, 1, g + (5,))
    # the agent lies 2 cells to the right and 1 cell up of the ego: the ego
    # cell (i, j) pulls the agent cell (i - 1, j - 2)
    out = N.warp(X, (0.0, 2 * dx, 1 * dy), cfg, g)
    want = np.zeros_like(X)
    want[1:, 2:] = X[:-1, :-2]
    np.testing.assert_allclose(out, want, atol=1e-12)


@pytest.mark.parametrize("name", ["t_attn", "t_max"])
def test_multiscale_one_agent_equals_single_scale(name):
    """One agent at the identity pose: fusing before or after upsampling is
    the same (fusion of one map returns it), so both shapes give exactly
    the same fused map and head output."""
    cfg = dict(synth.config(name), K=1)
    fr = synth.make_frame(name)
    fr1 = dict(fr, cfg=cfg, points=fr["points"][:1], poses=np.zeros((1, 3)))
    a = N.forward(fr1)
    b = N.forward(dict(fr1, cfg=_multiscale(cfg)))
    assert np.array_equal(a["fused"], b["fused"])
    assert np.array_equal(a["head"], b["head"])


def test_multiscale_max_of_identical_agents_is_one_agent():
    cfg = synth.config("t_max")
    fr = synth.make_frame(cfg)
    one = dict(cfg, K=1, multiscale=True)
    three = dict(cfg, K=3, multiscale=True)
    p0 = fr["points"][0]
    a = N.forward(dict(fr, cfg=one, points=[p0], poses=np.zeros((1, 3))))
    b = N.forward(dict(fr, cfg=three, points=[p0, p0, p0], poses=np.zeros((3, 3))))
    assert np.array_equal(a["fused"], b["fused"])
    for s in range(3):
        assert np.array_equal(a["fused_stages"][s], b["fused_stages"][s])


def test_multiscale_fuses_at_every_scale():
    """The scales are fused independently: the stage-s fused map is the
    fusion of the agents' warped stage-s maps, and the head reads the
    upsampled fused maps; with poses, fusing before upsampling differs
    from the single-scale shape (upsampling is not linear through ReLU)."""
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    ms = N.forward(dict(fr, cfg=_multiscale(cfg)), keep=True)
    for s, f in enumerate(ms["fused_stages"]):
        want = N._store(cfg, N.fuse_attn(ms["warped_stages"][s]))
        assert np.array_equal(f, want)
        assert f.shape[:2] == N.stage_grids(cfg)[s]
    assert ms["fused"].shape == N.forward(fr)["fused"].shape
    assert not np.array_equal(ms["fused"], N.forward(fr)["fused"])
