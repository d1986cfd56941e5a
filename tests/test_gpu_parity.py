"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Pillar cells and counts are compared bit for bit; activations by max-norm
relative error (1e-4 fp32, 2e-2 bf16); detections as sets with a tolerance
band around the threshold, before NMS; the NMS output exactly against the
oracle's NMS of the same decoded records.  RTCC and barrier runs of a frame
must give bitwise identical outputs."""

import sys

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R
from tests.helpers import (TOL, check_conv_layers, check_decode_exact, check_frame_nms, check_fusion_and_head,
                           check_members, compare_detections, make_ctx, rel_err, run_frame, tensors)

pytestmark = pytest.mark.gpu

_CACHE = {}


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _oracle(name):
    if name not in _CACHE:
        fr = synth.make_frame(name)
        _CACHE[name] = (fr, N.forward(fr, keep=True))
    return _CACHE[name]


def _check_frame(cfg, fr, ref, got, with_stages=True):
    tol = TOL[cfg["precision"]]
    K = cfg["K"]
    for k in range(K):
        e = ref["enc"][k]
        assert np.array_equal(got["cells"][k], e["cells"].astype(np.int32)), "pillar cells, agent %d" % k
        assert np.array_equal(got["counts"][k], e["counts"].astype(np.int32)), "pillar counts, agent %d" % k
        err = rel_err(got["canvas"][k], e["canvas"].ravel())
        assert err <= tol, ("canvas", k, err)
        if with_stages:
            for s, so in enumerate(e["stage_out"]):
                err = rel_err(got["stage"][k][s], so.ravel())
                assert err <= tol, ("stage", s, k, err)
        err = rel_err(got["slot"][k], e["slot"].ravel())
        assert err <= tol, ("slot", k, err)
    err = rel_err(got["fused"], ref["fused"].ravel())
    assert err <= tol, ("fused", err)
    err = rel_err(got["head"], ref["head"].ravel())
    assert err <= tol, ("head", err)


@pytest.mark.parametrize("name", ["t_max", "t_attn", "c1", "c2", "c3"])
def test_frame_parity_and_mode_identity(name):
    _say("parity %s" % name)
    cfg = synth.config(name)
    fr, ref = _oracle(name)
    with make_ctx(cfg, fr) as ctx:
        a = synth.arrival_draws(cfg, 1)[0] * 1e-3 if cfg["arrivals"]["kind"] != "uplink" else None
        det_r = run_frame(ctx, fr, R.RTCC_MODE_RELEASE, a)
        got_r = tensors(ctx, cfg)
        _check_frame(cfg, fr, ref, got_r)
        dec_r = check_frame_nms(ctx, det_r, cfg)
        compare_detections(dec_r, ref["det"], cfg, ref["head"])
        _say("  %s: %d decoded, %d after NMS" % (name, det_r["count_decoded"], det_r["count"]))
        # one kernel at a time, on the GPU's own inputs
        for k in range(cfg["K"]):
            check_members(ctx, cfg, fr["points"][k], k)
        pw = N.prepared_weights(cfg, fr["weights"])
        check_conv_layers(ctx, cfg, pw, 0)
        check_fusion_and_head(ctx, cfg, fr["poses"], pw)
        assert check_decode_exact(ctx, cfg) == det_r["count_decoded"]
        det_b = run_frame(ctx, fr, R.RTCC_MODE_BARRIER, a)
        got_b = tensors(ctx, cfg)
        dec_b = R.decoded_records(ctx)
    # RTCC and barrier: bitwise identical outputs and identical box sets
    for key in ("canvas", "slot"):
        for k in range(cfg["K"]):
            assert np.array_equal(got_r[key][k].view(np.uint32), got_b[key][k].view(np.uint32))
    assert np.array_equal(got_r["fused"].view(np.uint32), got_b["fused"].view(np.uint32))
    assert np.array_equal(got_r["head"].view(np.uint32), got_b["head"].view(np.uint32))
    assert np.array_equal(det_r["anchor_idx"], det_b["anchor_idx"])
    assert np.array_equal(det_r["boxes"].view(np.uint32), det_b["boxes"].view(np.uint32))
    assert np.array_equal(dec_r["anchor_idx"], dec_b["anchor_idx"])
    assert np.array_equal(dec_r["boxes"].view(np.uint32), dec_b["boxes"].view(np.uint32))


def test_repeated_frames_are_bitwise_identical():
    cfg = synth.config("t_attn")
    fr, _ref = _oracle("t_attn")
    with make_ctx(cfg, fr) as ctx:
        outs = []
        for _ in range(3):
            run_frame(ctx, fr)
            outs.append(tensors(ctx, cfg, with_stages=False))
    for o in outs[1:]:
        assert np.array_equal(o["fused"].view(np.uint32), outs[0]["fused"].view(np.uint32))
        assert np.array_equal(o["head"].view(np.uint32), outs[0]["head"].view(np.uint32))


def test_serial_executor_matches_per_branch_streams():
    cfg = synth.config("t_max")
    fr, _ref = _oracle("t_max")
    with make_ctx(cfg, fr) as a:
        run_frame(a, fr)
        ta = tensors(a, cfg, with_stages=False)
    with make_ctx(cfg, fr, exec=R.RTCC_EXEC_SERIAL) as b:
        run_frame(b, fr)
        tb = tensors(b, cfg, with_stages=False)
    assert np.array_equal(ta["head"].view(np.uint32), tb["head"].view(np.uint32))


def _edge_frame():
    """t_max frame with adversarial inputs: an empty agent, one cell holding
    500 points (cap 32), points on cell edges and range limits, NaN/Inf."""
    cfg = synth.config("t_max")
    fr = synth.make_frame(cfg)
    pts = [p.copy() for p in fr["points"]]
    pts[0] = np.zeros((0, 4), dtype=np.float32)
    p1 = pts[1]
    p1[:500, 0] = 0.1
    p1[:500, 1] = -0.3
    p1[500:520, 0] = np.float32(cfg["x_range"][1])           # x = xmax: dropped
    p1[520:540, 0] = np.float32(cfg["x_range"][0])           # x = xmin: kept
    p1[540:560, 1] = np.float32(-8.8) + np.float32(0.4) * 3  # near a row edge
    p1[560:570, 2] = np.nan
    p1[570:580, 3] = np.inf
    p1[580:590, 2] = np.float32(cfg["z_range"][1])           # z = zmax: dropped
    fr["points"] = pts
    return cfg, fr


def test_edge_cases_empty_agent_overfull_cell_and_invalid_points():
    cfg, fr = _edge_frame()
    ref = N.forward(fr, keep=True)
    assert ref["enc"][1]["counts"].max() >= 500
    with make_ctx(cfg, fr, max_points=cfg["n_points"]) as ctx:
        run_frame(ctx, fr)
        got = tensors(ctx, cfg)
        # which 32 of the 500 points fed the PFN, bit-exact
        assert check_members(ctx, cfg, fr["points"][0], 0) == 0
        check_members(ctx, cfg, fr["points"][1], 1)
        check_members(ctx, cfg, fr["points"][2], 2)
    assert got["cells"][0].size == 0 and got["counts"][0].size == 0
    _check_frame(cfg, fr, ref, got)


def test_max_points_exactly_and_ragged_tail():
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    # a point count that is not a multiple of any block size
    fr["points"] = [p[:4999 - 7 * k] for k, p in enumerate(fr["points"])]
    ref = N.forward(fr, keep=True)
    with make_ctx(cfg, fr, max_points=4999) as ctx:
        run_frame(ctx, fr)
        got = tensors(ctx, cfg)
    _check_frame(cfg, fr, ref, got)


def test_consecutive_frames_with_different_points_match_oracle():
    """No memset of the cell counts per frame (the PFN kernel returns them to
    zero): frames of different point sets on one context, one of them with a
    500-point cell and an empty agent, each match the oracle."""
    cfg, fr_e = _edge_frame()
    ref_e = N.forward(fr_e, keep=True)
    fr_n, ref_n = _oracle("t_max")
    with make_ctx(cfg, fr_e, max_points=cfg["n_points"]) as ctx:
        for i, (fr, ref) in enumerate(((fr_n, ref_n), (fr_e, ref_e), (fr_n, ref_n), (fr_e, ref_e))):
            _say("  frame %d" % i)
            run_frame(ctx, fr)
            _check_frame(cfg, fr, ref, tensors(ctx, cfg), with_stages=False)
            for k in range(cfg["K"]):
                check_members(ctx, cfg, fr["points"][k], k)


def test_branch_states_follow_the_device():
    """RELEASED at release, FINISHED once the device has run the encoder, read
    without a join (eq. branch_state)."""
    import time
    import torch
    cfg = synth.config("t_attn")
    fr, _ref = _oracle("t_attn")
    with make_ctx(cfg, fr) as ctx:
        R.rtcc_set_mode(ctx, R.RTCC_MODE_BARRIER)
        R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
        for k in range(cfg["K"] - 1):
            R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
            assert R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING
        k = cfg["K"] - 1
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
        assert all(R.rtcc_get_branch_state(ctx, j) >= R.RTCC_RELEASED for j in range(cfg["K"]))
        torch.cuda.synchronize()
        assert all(R.rtcc_get_branch_state(ctx, j) == R.RTCC_FINISHED for j in range(cfg["K"]))
        R.rtcc_join_and_detect(ctx)
        assert all(R.rtcc_get_branch_state(ctx, j) == R.RTCC_FINISHED for j in range(cfg["K"]))


@pytest.mark.parametrize("variant", [1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12])
@pytest.mark.parametrize("splits", [0, 2])
def test_forced_conv_tilings(variant, splits):
    """Each 3x3-conv tiling (and split-K) forced on every layer it supports,
    on a grid with several ragged tiles per layer at c5's channel counts:
    every layer elementwise against the oracle conv of its GPU input, and
    the head against the oracle end to end."""
    _say("forced conv tiling %d splits %d" % (variant, splits))
    cfg = synth.config("t_var")
    fr, ref = _oracle("t_var")
    with make_ctx(cfg, fr, conv_variant=variant, conv_splits=splits) as ctx:
        run_frame(ctx, fr)
        plans = [R.rtcc_conv_plan(ctx, l) for l in range(sum(n for _s, _c, n in cfg["stages"]))]
        _say("  plans %s" % plans)
        want = 0 if variant == 7 else variant
        assert sum(v == want for v, _sp in plans) >= 1
        if splits:
            assert any(sp == splits for _v, sp in plans) or variant in (5, 6)
        pw = N.prepared_weights(cfg, fr["weights"])
        for k in range(cfg["K"]):
            check_conv_layers(ctx, cfg, pw, k)
        got = tensors(ctx, cfg)
    _check_frame(cfg, fr, ref, got)


def test_torch_allocator_and_stream_hook():
    """Device buffers from PyTorch's caching allocator and the post-join
    subgraph on a torch stream give the same frame, bit for bit."""
    import torch
    cfg = synth.config("t_attn")
    fr, _ref = _oracle("t_attn")
    with make_ctx(cfg, fr) as ctx:
        run_frame(ctx, fr)
        want = tensors(ctx, cfg, with_stages=False)
    before = torch.cuda.memory_allocated()
    st = torch.cuda.Stream()
    with make_ctx(cfg, fr, torch_memory=True, join_stream=st) as ctx:
        assert torch.cuda.memory_allocated() > before
        for _ in range(2):
            run_frame(ctx, fr)
            got = tensors(ctx, cfg, with_stages=False)
            assert np.array_equal(got["head"].view(np.uint32), want["head"].view(np.uint32))
            assert np.array_equal(got["fused"].view(np.uint32), want["fused"].view(np.uint32))
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before


def test_frame_after_an_infeasible_frame_matches_oracle():
    """An infeasible frame runs some encoders but no join, so their canvas
    pillars are not cleared after it: the next encoder of each branch clears
    them first, and the next frame (other points) matches the oracle."""
    import time
    cfg, fr_e = _edge_frame()
    fr_n, ref_n = _oracle("t_max")
    with make_ctx(cfg, fr_e, max_points=cfg["n_points"]) as ctx:
        run_frame(ctx, fr_e)
        R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
        for k in range(cfg["K"] - 1):
            R.rtcc_release_branch(ctx, k, fr_n["points"][k], fr_n["poses"][k], 0.0)
        with pytest.raises(R.RtccError) as e:
            R.rtcc_join_and_detect(ctx)
        assert e.value.status == R.RTCC_E_INFEASIBLE
        run_frame(ctx, fr_n)
        _check_frame(cfg, fr_n, ref_n, tensors(ctx, cfg), with_stages=False)
        for k in range(cfg["K"]):
            check_members(ctx, cfg, fr_n["points"][k], k)


@pytest.mark.parametrize("graphs", [0, 1])
def test_join_reads_back_more_records_than_the_first_block(graphs):
    """With NMS off and a threshold below every logit, the join returns every
    anchor of c1 (8,192, more than the 1,024 records the last kernel of the
    join writes to host memory; the rest come by copy).  Three frames in a
    row (the join clears the export flag and waits for it again each time),
    each bit for bit the GPU's own decoded records, which match the oracle's
    decode of the GPU's head output."""
    _say("join read-back beyond the first records, graphs %d" % graphs)
    cfg = synth.config("c1")
    cfg["nms_max_candidates"] = 0
    cfg["logit_threshold"] = -1e30
    fr, _ref = _oracle("c1")
    with make_ctx(cfg, fr, use_graphs=graphs) as ctx:
        for _ in range(3):
            det = run_frame(ctx, fr)
            n = check_decode_exact(ctx, cfg)
            dec = R.decoded_records(ctx)
            assert det["count"] == det["count_decoded"] == n > 1024
            assert np.array_equal(det["anchor_idx"], dec["anchor_idx"])
            assert np.array_equal(det["boxes"].view(np.uint32), dec["boxes"].view(np.uint32))
            assert np.array_equal(det["scores"].view(np.uint32), dec["scores"].view(np.uint32))
