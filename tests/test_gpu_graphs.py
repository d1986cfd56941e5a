"""HIP graphs (use_graphs = 1): a context that replays its branches and its
join as graphs gives bitwise the outputs of an eager context on the same
frames.  The frame sequence repeats inputs (plain replays), changes point
counts and poses (graphs updated in place, or launched eagerly for a
frame whose arguments differ from its predecessor's) and alternates RTCC
and barrier;
torch runs its own kernels, and both sides synchronize, between frames, and
every frame of the graph context is checked against the eager one."""

import sys

import numpy as np
import pytest
import torch

import synth
from paper_2608_08330_amd import rtcc as R
from tests.helpers import make_ctx, run_frame

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _frames(fr, K):
    """(points, poses, mode) of each frame: repeats, fewer points, moved poses."""
    pts, poses = fr["points"], np.asarray(fr["poses"], dtype=np.float64)
    moved = poses.copy()
    moved[1:, 0] += 0.75
    moved[1:, 2] += 0.05
    fewer = [p[:max(1, len(p) - 37 * (k + 1))] for k, p in enumerate(pts)]
    seq = [(pts, poses, R.RTCC_MODE_RELEASE)] * 3
    seq += [(fewer, poses, R.RTCC_MODE_BARRIER), (fewer, poses, R.RTCC_MODE_RELEASE)]
    seq += [(pts, moved, R.RTCC_MODE_RELEASE)] * 2
    seq += [(pts, poses, R.RTCC_MODE_BARRIER)] * 2
    return seq


def _outputs(ctx, cfg, det):
    out = dict(fused=R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED, 0, np.uint8),
               head=R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.uint8),
               idx=np.array(det["anchor_idx"]), boxes=np.array(det["boxes"]).view(np.uint32),
               scores=np.array(det["scores"]).view(np.uint32), decoded=det["count_decoded"])
    for k in range(cfg["K"]):
        out["cells%d" % k] = R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_CELLS, k, np.int32)
        if cfg.get("warp_in_branch"):
            out["warped%d" % k] = R.rtcc_get_tensor(ctx, R.RTCC_T_WARPED, k, np.uint8)
    if cfg.get("multiscale"):
        for s in range(len(cfg["stages"])):
            out["stage%d" % s] = R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED_STAGE, s, np.uint8)
    return out


def _torch_work():
    x = torch.randn(512, 512, device="cuda")
    y = (x @ x).relu_().sum()
    torch.cuda.synchronize()
    return float(y)


CASES = [("t_attn", "streams", {}), ("t_max", "serial", {}), ("c2", "streams", {}),
         ("c1", "streams", {"warp_in_branch": True}), ("t_attn", "serial", {"multiscale": True})]


@pytest.mark.parametrize("name,exec_kind,extra", CASES, ids=["%s-%s-%s" % (n, e, "-".join(x) or "plain")
                                                            for n, e, x in CASES])
def test_graph_replays_equal_eager(name, exec_kind, extra):
    cfg = dict(synth.config(name), **extra)
    fr = dict(synth.make_frame(name), cfg=cfg)
    ex = R.RTCC_EXEC_SERIAL if exec_kind == "serial" else R.RTCC_EXEC_PER_BRANCH_STREAMS
    K = cfg["K"]
    seq = _frames(fr, K)
    _say("graphs %s %s %s: %d frames" % (name, exec_kind, extra, len(seq)))
    with make_ctx(cfg, fr, exec=ex) as eager, make_ctx(cfg, fr, exec=ex, use_graphs=1) as graph:
        assert R.rtcc_graph_stats(graph) == (0, 0, 0)
        for i, (pts, poses, mode) in enumerate(seq):
            f = dict(fr, points=pts, poses=poses)
            want = _outputs(eager, cfg, run_frame(eager, f, mode))
            _torch_work()
            got = _outputs(graph, cfg, run_frame(graph, f, mode))
            _torch_work()
            for key in want:
                assert np.array_equal(np.asarray(want[key]), np.asarray(got[key])), (i, key)
            assert want["decoded"] > 0 or name.startswith("t_"), i
        inst, upd, launches = R.rtcc_graph_stats(graph)
        assert R.rtcc_graph_stats(eager) == (0, 0, 0)
    # Graphs: every branch's backbone and (released alone) pillar stage, a
    # group's two, and the join's two.  The backbones and the detection
    # graph replay every frame; the pillar stages and the fusion are replayed
    # only where a frame repeats its predecessor's arguments (otherwise
    # launched eagerly), and a changed argument updates a graph in place
    # rather than instantiating another.
    n_bar = sum(1 for _p, _q, m in seq if m == R.RTCC_MODE_BARRIER)
    assert launches >= (len(seq) - n_bar) * (K + 1) + n_bar * 2
    assert inst <= 2 * K + 4
    assert upd >= 1
    _say("  instantiated %d, updates %d, launches %d" % (inst, upd, launches))


def test_graphs_are_off_while_node_timing():
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    with make_ctx(cfg, fr, use_graphs=1, node_timing=1) as ctx:
        run_frame(ctx, fr)
        assert R.rtcc_graph_stats(ctx) == (0, 0, 0)
        assert sum(R.rtcc_node_times(ctx)) > 0
