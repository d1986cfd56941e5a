"""Full-size c5 parity (8 agents x 100,000 points, 512 x 512 BEV, bf16,
attention fusion), every tensor compared in full, in the launch
configuration bench.py times for its roofline pass (one compute stream,
device-resident inputs).

Two kinds of comparison:
  * one kernel at a time: the oracle op applied to the GPU's own input of
    that op (every conv layer and upsampling of three agents, the warp +
    fusion, the head, the decode), elementwise within one bf16 rounding
    step; a tile-edge or XCD-band error shows as a single element;
  * end to end: the oracle network run from the points (every agent's
    pillars, members, canvas, stage outputs and slot, then the fused map,
    head and detections), within the bf16 bar of 2e-2 max-norm relative.
The multi-scale fusion network runs on the same frame and is checked both
ways too."""

import sys
import time

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R
from tests.helpers import (BF16_STEP, TOL, as_f32, assert_close_elementwise, check_conv_layers,
                           check_decode_exact, check_fusion_and_head, check_members, compare_detections,
                           make_ctx, rel_err)

pytestmark = pytest.mark.gpu

_ORACLE = {}  # agent -> oracle encoder output (keep=True)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _release_all(ctx, cfg, fr, dev):
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
    for k in range(cfg["K"]):
        R.rtcc_release_branch_device(ctx, k, dev[k].data_ptr(), len(fr["points"][k]), fr["poses"][k], 0.0)
    return R.rtcc_join_and_detect(ctx)


@pytest.fixture(scope="module")
def c5():
    import torch
    _say("c5 full: GPU frame")
    cfg = synth.config("c5")
    fr = synth.make_frame(cfg)
    dev = [torch.from_numpy(p).to("cuda") for p in fr["points"]]
    torch.cuda.synchronize()
    ctx = make_ctx(cfg, fr, exec=R.RTCC_EXEC_SERIAL)
    det = _release_all(ctx, cfg, fr, dev)
    pw = N.prepared_weights(cfg, fr["weights"])
    yield dict(cfg=cfg, fr=fr, ctx=ctx, det=det, pw=pw, dev=dev)
    ctx.close()


def _oracle_encoder(c5, k):
    if k not in _ORACLE:
        _ORACLE[k] = N.encoder(c5["fr"]["points"][k], c5["cfg"], c5["pw"], keep=True)
    return _ORACLE[k]


def test_c5_pillars_members_and_canvas(c5):
    cfg, fr, ctx = c5["cfg"], c5["fr"], c5["ctx"]
    H, W = N.grid(cfg)
    for k in range(cfg["K"]):
        _say("  agent %d pillars" % k)
        pil = N.pillars(N.cell_ids(fr["points"][k], cfg), cfg["max_pts"])
        assert np.array_equal(R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_CELLS, k, np.int32),
                              pil["cells"].astype(np.int32))
        assert np.array_equal(R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_COUNTS, k, np.int32),
                              pil["counts"].astype(np.int32))
        check_members(ctx, cfg, fr["points"][k], k)
        canvas = N._store(cfg, N.pfn_canvas(fr["points"][k], pil, c5["pw"]["pfn_w"], c5["pw"]["pfn_b"], cfg))
        got = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_CANVAS, k), cfg).reshape(H, W, -1)
        assert_close_elementwise(got, canvas, BF16_STEP, 1e-4, ("canvas", k))


@pytest.mark.parametrize("agent", [0, 3, 7])
def test_c5_every_conv_layer_and_upsampling(c5, agent):
    _say("  agent %d: 13 conv layers + 3 upsamplings, one at a time" % agent)
    errs = check_conv_layers(c5["ctx"], c5["cfg"], c5["pw"], agent)
    _say("  max deviation per layer / max: %s" % ["%.1e" % e for e in errs])


def test_c5_conv_plan(c5):
    """The tilings the planner gives the 13 c5 layers (256 CUs): the
    64-channel stride-2 entry as the implicit GEMM with 256-pixel tiles,
    stage 0 as 8-row
    tiles, the stage-1 entry as 8-row stride-2 tiles, stage 1 as 8-row tiles
    with 64-byte channel chunks, the stage-2 entry and stage 2 as 4-row
    tiles (their batched launches take the 8-row forms of the same
    accumulation order); no layer split over its K loop."""
    plans = [R.rtcc_conv_plan(c5["ctx"], l) for l in range(13)]
    _say("  plans %s" % plans)
    assert plans == [(v, 1) for v in (12, 1, 1, 3, 8, 8, 8, 8, 4, 2, 2, 2, 2)]


def test_c5_fusion_head_and_decode(c5):
    _say("  warp + attention fusion, head, decode")
    e_f, e_h = check_fusion_and_head(c5["ctx"], c5["cfg"], c5["fr"]["poses"], c5["pw"])
    n = check_decode_exact(c5["ctx"], c5["cfg"])
    assert n == c5["det"]["count_decoded"] and n > 0
    _say("  fusion %.1e, head %.1e, %d decoded" % (e_f, e_h, n))


@pytest.mark.parametrize("agent", range(8))
def test_c5_encoder_end_to_end(c5, agent):
    """Agent k's encoder from its points: every stage output and the slot in
    full against the oracle network."""
    cfg, ctx = c5["cfg"], c5["ctx"]
    tol = TOL["bf16"]
    _say("  agent %d end to end" % agent)
    e = _oracle_encoder(c5, agent)
    for s, so in enumerate(e["stage_out"]):
        got = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_STAGE_OUT, (s << 8) | agent), cfg)
        err = rel_err(got, so.ravel())
        assert err <= tol, ("stage", s, err)
    err = rel_err(as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_SLOT, agent), cfg), e["slot"].ravel())
    assert err <= tol, ("slot", err)


def test_c5_fused_head_detections_end_to_end(c5):
    cfg, fr, ctx = c5["cfg"], c5["fr"], c5["ctx"]
    tol = TOL["bf16"]
    slots = [_oracle_encoder(c5, k)["slot"] for k in range(cfg["K"])]
    warped = [N.warp(slots[k], fr["poses"][k], cfg) for k in range(cfg["K"])]
    fused = N._store(cfg, N.fuse_attn(warped))
    Z = N.head(fused, c5["pw"]["head_w"], c5["pw"]["head_b"])
    err_f = rel_err(as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg), fused.ravel())
    err_h = rel_err(R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32), Z.ravel())
    _say("  end to end: fused %.2e, head %.2e" % (err_f, err_h))
    assert err_f <= tol and err_h <= tol
    compare_detections(R.decoded_records(ctx), N.decode(Z, cfg), cfg, Z)


def test_c5_multiscale(c5):
    """Multi-scale fusion on the same frame: each scale's fused map against
    the oracle warp + fusion of the GPU's stage outputs, the upsampled
    concatenation against the oracle upsampling of the GPU's fused maps
    (elementwise), then the whole network end to end (2e-2)."""
    cfg = dict(c5["cfg"], multiscale=True)
    fr, pw = c5["fr"], c5["pw"]
    tol = TOL["bf16"]
    grids = N.stage_grids(cfg)
    H2, W2 = N.feature_grid(cfg)
    up = cfg["up_channels"]
    frm = dict(fr, cfg=cfg)
    with make_ctx(cfg, frm, exec=R.RTCC_EXEC_SERIAL) as ctx:
        _release_all(ctx, cfg, fr, c5["dev"])
        fused_cat = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg).reshape(H2, W2, -1)
        head = R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32).reshape(H2, W2, 16)
        rel_u = 1
        oracle_parts = []
        for s, (stride, c, _n) in enumerate(cfg["stages"]):
            if s > 0:
                rel_u *= stride
            Hs, Ws = grids[s]
            _say("  multi-scale stage %d (%d x %d)" % (s, Hs, Ws))
            maps = [as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_STAGE_OUT, (s << 8) | k), cfg).reshape(Hs, Ws, c)
                    .astype(np.float64) for k in range(cfg["K"])]
            f_ref = N._store(cfg, N.fuse_attn([N.warp(maps[k], fr["poses"][k], cfg, grids[s])
                                               for k in range(cfg["K"])]))
            f_gpu = as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED_STAGE, s), cfg).reshape(Hs, Ws, c)
            assert_close_elementwise(f_gpu, f_ref, BF16_STEP, 1e-3, ("fused stage", s))
            u_ref = N._store(cfg, N.deconv(f_gpu.astype(np.float64), pw["up%d_w" % s], pw["up%d_b" % s], rel_u,
                                           H2, W2))
            assert_close_elementwise(fused_cat[:, :, s * up:(s + 1) * up], u_ref, BF16_STEP, 1e-4, ("upsample", s))
            # end to end: the oracle's own stage outputs of every agent
            enc = [_oracle_encoder(c5, k)["stage_out"][s] for k in range(cfg["K"])]
            f_e2e = N._store(cfg, N.fuse_attn([N.warp(enc[k], fr["poses"][k], cfg, grids[s])
                                               for k in range(cfg["K"])]))
            assert rel_err(f_gpu.ravel(), f_e2e.ravel()) <= tol, ("fused stage end to end", s)
            oracle_parts.append(N._store(cfg, N.deconv(f_e2e, pw["up%d_w" % s], pw["up%d_b" % s], rel_u, H2, W2)))
        head_ref = N.head(fused_cat.astype(np.float64), pw["head_w"], pw["head_b"])
        assert_close_elementwise(head, head_ref, 1e-5, 1e-5, "multi-scale head")
        Z = N.head(np.concatenate(oracle_parts, axis=2), pw["head_w"], pw["head_b"])
        err = rel_err(head, Z.ravel())
        _say("  multi-scale head end to end %.2e" % err)
        assert err <= tol
        n = check_decode_exact(ctx, cfg)
        _say("  multi-scale: %d decoded" % n)
