"""GPU parity of multi-scale fusion (multiscale = 1): every scale's fused
map, the upsampled concatenation, the head and the detections against the
oracle of the same shape; RTCC and barrier bitwise identical; one agent at
the identity pose gives bitwise the single-scale result."""

import sys

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R
from tests.helpers import TOL, as_f32, check_frame_nms, compare_detections, make_ctx, rel_err, run_frame

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _outputs(ctx, cfg):
    S = len(cfg["stages"])
    return dict(
        stages=[as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED_STAGE, s), cfg) for s in range(S)],
        fused=as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg),
        head=R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32),
    )


@pytest.mark.parametrize("name", ["t_attn", "t_max", "c2", "c3"])
def test_multiscale_parity_and_mode_identity(name):
    _say("multiscale parity %s" % name)
    cfg = dict(synth.config(name), multiscale=True)
    fr = dict(synth.make_frame(name), cfg=cfg)
    ref = N.forward(fr)
    tol = TOL[cfg["precision"]]
    a = synth.arrival_draws(cfg, 1)[0] * 1e-3 if cfg["arrivals"]["kind"] != "uplink" else None
    with make_ctx(cfg, fr) as ctx:
        det_r = run_frame(ctx, fr, R.RTCC_MODE_RELEASE, a)
        got_r = _outputs(ctx, cfg)
        for s, f in enumerate(ref["fused_stages"]):
            assert rel_err(got_r["stages"][s], f.ravel()) <= tol, ("fused stage", s)
        assert rel_err(got_r["fused"], ref["fused"].ravel()) <= tol
        assert rel_err(got_r["head"], ref["head"].ravel()) <= tol
        dec_r = check_frame_nms(ctx, det_r, cfg)
        compare_detections(dec_r, ref["det"], cfg, ref["head"])
        with pytest.raises(R.RtccError):
            R.rtcc_get_tensor(ctx, R.RTCC_T_SLOT, 0)
        _say("  %s: %d decoded, %d after NMS" % (name, det_r["count_decoded"], det_r["count"]))
        det_b = run_frame(ctx, fr, R.RTCC_MODE_BARRIER, a)
        got_b = _outputs(ctx, cfg)
    for key in ("fused", "head"):
        assert np.array_equal(got_r[key].view(np.uint32), got_b[key].view(np.uint32))
    for s in range(len(cfg["stages"])):
        assert np.array_equal(got_r["stages"][s].view(np.uint32), got_b["stages"][s].view(np.uint32))
    assert np.array_equal(det_r["anchor_idx"], det_b["anchor_idx"])
    assert np.array_equal(det_r["boxes"].view(np.uint32), det_b["boxes"].view(np.uint32))


@pytest.mark.parametrize("name", ["t_attn", "t_max"])
def test_one_agent_multiscale_equals_single_scale(name):
    out = {}
    for ms in (False, True):
        cfg = dict(synth.config(name), K=1, multiscale=ms)
        fr = synth.make_frame(name)
        fr = dict(fr, cfg=cfg, points=fr["points"][:1], poses=np.zeros((1, 3)))
        with make_ctx(cfg, fr) as ctx:
            run_frame(ctx, fr)
            out[ms] = (as_f32(R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED), cfg),
                       R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.float32))
    for i in range(2):
        assert np.array_equal(out[False][i].view(np.uint32), out[True][i].view(np.uint32))


def test_c5_multiscale_mode_identity():
    _say("multiscale c5")
    cfg = dict(synth.config("c5"), multiscale=True)
    fr = dict(synth.make_frame("c5"), cfg=cfg)
    a = synth.arrival_draws(cfg, 1)[0] * 1e-3
    with make_ctx(cfg, fr) as ctx:
        det_r = run_frame(ctx, fr, R.RTCC_MODE_RELEASE, a)
        got_r = _outputs(ctx, cfg)
        det_b = run_frame(ctx, fr, R.RTCC_MODE_BARRIER, a)
        got_b = _outputs(ctx, cfg)
    assert np.array_equal(got_r["head"].view(np.uint32), got_b["head"].view(np.uint32))
    assert np.array_equal(det_r["anchor_idx"], det_b["anchor_idx"])
    assert det_r["count"] > 0
