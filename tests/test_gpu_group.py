"""Branches released together (rtcc_release_branches, and every branch at
the barrier's A) share one pillar-stage launch chain over the group (one
grid row per agent), after which each backbone runs on its own stream.  The
outputs must equal those of separate releases bit for bit: pillar lists and
counts, used members, canvas, slots, fused map, head and detections; and a
group frame must match the oracle."""

import sys
import time

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R
from tests.helpers import TOL, make_ctx, rel_err, run_frame, tensors

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _host_events(fr, agents):
    return [dict(agent=k, points=fr["points"][k], pose=fr["poses"][k], arrival_t=0.0) for k in agents]


def _run_batches(ctx, fr, batches, mode=R.RTCC_MODE_RELEASE, events=_host_events):
    R.rtcc_set_mode(ctx, mode)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
    for b in batches:
        st = []
        R.rtcc_release_branches(ctx, events(fr, b), st)
        assert st == [R.RTCC_OK] * len(b)
    return R.rtcc_join_and_detect(ctx)


def _raw(ctx, K):
    out = {}
    for k in range(K):
        for tid in (R.RTCC_T_PILLAR_CELLS, R.RTCC_T_PILLAR_COUNTS, R.RTCC_T_CANVAS, R.RTCC_T_SLOT):
            out[(tid, k)] = R.rtcc_get_tensor(ctx, tid, k, np.uint8)
        out[("members", k)] = R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_MEMBERS, k, np.int32)
    out["fused"] = R.rtcc_get_tensor(ctx, R.RTCC_T_FUSED, 0, np.uint8)
    out["head"] = R.rtcc_get_tensor(ctx, R.RTCC_T_HEAD, 0, np.uint8)
    return out


def _same(d0, r0, d1, r1, what):
    assert d0["count"] == d1["count"], what
    for key in ("anchor_idx", "boxes", "scores"):
        assert np.array_equal(d0[key], d1[key]), (what, key)
    assert r0.keys() == r1.keys()
    for key in r0:
        assert np.array_equal(r0[key], r1[key]), (what, key)


@pytest.mark.parametrize("name", ["t_max", "c1", "c3", "t_var"])
@pytest.mark.parametrize("graphs", [0, 1])
def test_group_release_equals_separate_releases(name, graphs):
    _say("group %s graphs=%d" % (name, graphs))
    cfg = synth.config(name)
    fr = synth.make_frame(cfg)
    K = cfg["K"]
    with make_ctx(cfg, fr, use_graphs=graphs) as ctx:
        d0 = run_frame(ctx, fr)
        r0 = _raw(ctx, K)
        for batches in ([list(range(K))[::-1]], [[1, 0], list(range(2, K))], [[k] for k in range(K)]):
            d1 = _run_batches(ctx, fr, batches)
            _same(d0, r0, d1, _raw(ctx, K), (name, batches))
        # barrier: the K-th event releases all K as one group
        d2 = run_frame(ctx, fr, mode=R.RTCC_MODE_BARRIER)
        _same(d0, r0, d2, _raw(ctx, K), (name, "barrier"))
        d3 = _run_batches(ctx, fr, [[0, 1], list(range(2, K))], mode=R.RTCC_MODE_BARRIER)
        _same(d0, r0, d3, _raw(ctx, K), (name, "barrier batches"))


def test_group_release_on_the_serial_executor():
    cfg = synth.config("c3")
    fr = synth.make_frame(cfg)
    K = cfg["K"]
    with make_ctx(cfg, fr) as a, make_ctx(cfg, fr, exec=R.RTCC_EXEC_SERIAL) as b:
        d0 = run_frame(a, fr)
        r0 = _raw(a, K)
        for graphs_ctx in (b,):
            d1 = _run_batches(graphs_ctx, fr, [list(range(K))])
            _same(d0, r0, d1, _raw(graphs_ctx, K), "serial")


def _edge_frame():
    """t_max frame with an empty agent and a 500-point cell (cap 32)."""
    cfg = synth.config("t_max")
    fr = synth.make_frame(cfg)
    pts = [p.copy() for p in fr["points"]]
    pts[0] = np.zeros((0, 4), dtype=np.float32)
    pts[1][:500, 0] = 0.1
    pts[1][:500, 1] = -0.3
    pts[2] = pts[2][:777]  # a short, ragged agent beside a full one
    fr["points"] = pts
    return cfg, fr


def test_group_with_an_empty_agent_and_an_overfull_cell_matches_oracle():
    cfg, fr = _edge_frame()
    ref = N.forward(fr, keep=True)
    K = cfg["K"]
    with make_ctx(cfg, fr, max_points=cfg["n_points"]) as ctx:
        d0 = run_frame(ctx, fr)
        r0 = _raw(ctx, K)
        d1 = _run_batches(ctx, fr, [list(range(K))])
        r1 = _raw(ctx, K)
        got = tensors(ctx, cfg)
    _same(d0, r0, d1, r1, "edge")
    tol = TOL[cfg["precision"]]
    for k in range(K):
        e = ref["enc"][k]
        assert np.array_equal(got["cells"][k], e["cells"].astype(np.int32)), k
        assert np.array_equal(got["counts"][k], e["counts"].astype(np.int32)), k
        assert rel_err(got["canvas"][k], e["canvas"].ravel()) <= tol
        assert rel_err(got["slot"][k], e["slot"].ravel()) <= tol
    assert rel_err(got["head"], ref["head"].ravel()) <= tol


def test_c5_device_group_equals_separate_device_releases():
    """The benchmark's release: the 8 c5 agents' device-resident inputs in
    one batch, graphs on, over two stream frames."""
    import torch
    cfg = synth.config("c5")
    K = cfg["K"]
    frames = [synth.make_frame(cfg, f) for f in range(2)]
    dev = [[torch.from_numpy(p).to("cuda") for p in fr["points"]] for fr in frames]
    torch.cuda.synchronize()

    def dev_events(fi):
        def ev(fr, agents):
            return [dict(agent=k, device=1, points=dev[fi][k].data_ptr(), n=len(fr["points"][k]),
                         pose=fr["poses"][k], arrival_t=0.0) for k in agents]
        return ev

    with make_ctx(cfg, frames[0], use_graphs=1) as ctx:
        for fi, fr in enumerate(frames):
            _say("c5 group frame %d" % fi)
            R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
            R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
            for k in range(K):
                R.rtcc_release_branch_device(ctx, k, dev[fi][k].data_ptr(), len(fr["points"][k]), fr["poses"][k], 0.0)
            d0 = R.rtcc_join_and_detect(ctx)
            r0 = _raw(ctx, K)
            d1 = _run_batches(ctx, fr, [list(range(K))], events=dev_events(fi))
            _same(d0, r0, d1, _raw(ctx, K), ("c5", fi))
        s = R.rtcc_graph_stats(ctx)
        assert s[2] > 0
